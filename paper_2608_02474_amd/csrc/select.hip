// Saliency and recompute selection (Sec. 3.1 Eq. 1, applied per token against
// its cached input; Sec. 3.3 saliency mask with k = ceil(r L) tokens).
//
// saliency_rows: one wave per token row loads x and xref with 16-byte
//   non-temporal loads (all of a lane's loads issued before the first is
//   used) and accumulates
//   |x - xref| and |xref| in fp64 (exact per-element differences, so only the
//   summation order differs from the definition).
//   Writes s_i = fp32(w_frame * num / (den + xi)) plus num/den for the step sum.
// step_delta_sum: step-level Eq. 1 sum in a fixed order (deterministic); in
//   echo_select the same sum runs as a second workgroup of select_rows.
// select_rows: one 1024-thread workgroup, the keys held in registers
//   (1) top-K threshold key by 4-pass 8-bit radix select over order-preserving
//       uint32 keys (histograms in LDS);
//   (2) stable compaction in index order: per (1024-key round, wave) counts,
//       two block-wide exclusive scans (ranks of equal keys, output slots),
//       then wave ballot + popcount within each wave; ties at the threshold
//       key go to the lowest indices.
// The key set is tiny (4 bytes per token, L2-resident), so one workgroup keeps
// the selection exact and deterministic at a cost of a few microseconds.
// select_segments: the same selection per anchor segment, one workgroup per
//   segment (the two-stage form: anchor segments, then min(k, N) tokens each).
// anchor_select: the anchor segments (top-k of per-segment keys, or evenly
//   spaced), one workgroup.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kSalThreads = 256;
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

// MAXC > 0: a lane's MAXC chunks of 8 elements of x and xref are all loaded
// before any is used (D <= 512 MAXC); MAXC == 0 streams the row (any D).
template <typename T, int MAXC>
__global__ void __launch_bounds__(kSalThreads)
saliency_rows(const T* __restrict__ x, const T* __restrict__ xref, const float* __restrict__ fw,
              int L, int N, int D, double xi, float* __restrict__ s_out,
              double* __restrict__ num_out, double* __restrict__ den_out) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * (kSalThreads / kWave) + wave;
  if (row >= L) return;
  const T* xr = x + row * D;
  const T* rr = xref + row * D;
  const int nch = D / 8;
  double num = 0.0, den = 0.0;
  auto add8 = [&](const Raw8<T>& a, const Raw8<T>& b) __attribute__((always_inline)) {
    float fa[8], fb[8];
    a.unpack(fa);
    b.unpack(fb);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double da = fa[j], db = fb[j];
      num += fabs(da - db);
      den += fabs(db);
    }
  };
  if (MAXC > 0) {
    constexpr int R = MAXC > 0 ? MAXC : 1;
    Raw8<T> ra[R], rb[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int c = lane + u * kWave;
      const int cc = c < nch ? c : nch - 1;  // past the row end: in-bounds re-load, not added
      ra[u].load_nt(xr + cc * 8);
      rb[u].load_nt(rr + cc * 8);
    }
#pragma unroll
    for (int u = 0; u < R; ++u)
      if (lane + u * kWave < nch) add8(ra[u], rb[u]);
  } else {
    for (int c = lane; c < nch; c += kWave) {
      Raw8<T> a, b;
      a.load(xr + c * 8);
      b.load(rr + c * 8);
      add8(a, b);
    }
  }
  num = wave_sum(num);
  den = wave_sum(den);
  if (lane == 0) {
    const double delta = num / (den + xi);
    const double w = static_cast<double>(fw[row / N]);
    s_out[row] = __double2float_rn(w * delta);
    num_out[row] = num;
    den_out[row] = den;
  }
}

// Step-level Eq. 1 value sum(num) / (sum(den) + xi) in a fixed summation
// order (deterministic), by one 1024-thread workgroup: its own kernel after a
// saliency-only call, or the second workgroup of the select_rows launch.
__device__ __forceinline__ void step_delta_block(const double* __restrict__ num, const double* __restrict__ den,
                                                 int L, double xi, double* __restrict__ step_delta) {
  __shared__ double red_n[kSelWaves], red_d[kSelWaves];
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  double a = 0.0, b = 0.0;
  // unrolled so that eight loads of each array are in flight; the additions
  // keep their order
#pragma unroll 8
  for (int i = tid; i < L; i += kSelThreads) {
    a += num[i];
    b += den[i];
  }
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) {
    red_n[wave] = a;
    red_d[wave] = b;
  }
  __syncthreads();
  if (tid == 0) {
    double sa = 0.0, sb = 0.0;
    for (int w = 0; w < kSelWaves; ++w) {
      sa += red_n[w];
      sb += red_d[w];
    }
    *step_delta = sa / (sb + xi);
  }
}

__global__ void __launch_bounds__(kSelThreads)
step_delta_sum(const double* __restrict__ num, const double* __restrict__ den, int L, double xi,
               double* __restrict__ step_delta) {
  step_delta_block(num, den, L, xi, step_delta);
}

// Order-preserving key: larger float -> larger key; NaN above everything; -0 == +0.
__device__ __forceinline__ uint32_t rank_key(float s) {
  if (s != s) return 0xffffffffu;
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Top-k (or threshold) selection of L keys by one 1024-thread workgroup:
// writes mask[0..L), the selected positions i as idx_base + i in ascending
// order to idx[0..), and their number to *n_sel if n_sel is not null.
// R > 0: the L keys are loaded once into registers (key r*1024 + tid in
// slot r, L <= 1024 R), all loads in flight together; every later pass works
// on the registers.  R == 0: keys are re-read from s on every pass (any L).
template <int R>
__device__ __forceinline__ void topk_rows(const float* __restrict__ s, int L, int k, int threshold_mode,
                                          float threshold, int idx_base, int32_t* __restrict__ idx,
                                          uint8_t* __restrict__ mask, int32_t* __restrict__ n_sel) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_digit, sh_above;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const uint64_t lt_mask = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));

  constexpr int RR = R > 0 ? R : 1;
  uint32_t kr[RR];
  if constexpr (R > 0) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = r * kSelThreads + tid;
      kr[r] = i < L ? rank_key(s[i]) : 0u;
    }
  }
  const int nr = R > 0 ? R : (L + kSelThreads - 1) / kSelThreads;
  auto key_of = [&](int r, int i) __attribute__((always_inline)) -> uint32_t {
    if constexpr (R > 0)
      return kr[r];
    else
      return i < L ? rank_key(s[i]) : 0u;
  };

  // (1) threshold key and how many tokens equal to it are taken
  uint32_t thr;
  uint32_t need_eq;
  bool take_eq;
  if (threshold_mode) {
    thr = rank_key(threshold);
    need_eq = 0;
    take_eq = false;
  } else if (k == 0) {
    thr = 0xffffffffu;
    need_eq = 0;
    take_eq = true;
  } else {
    uint32_t prefix = 0, pmask = 0, kk = static_cast<uint32_t>(k);
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < (R > 0 ? R : 1); ++r) {
        for (int rr = (R > 0 ? r : 0); rr < (R > 0 ? r + 1 : nr); ++rr) {
          const int i = rr * kSelThreads + tid;
          const uint32_t key = key_of(rr, i);
          const bool in = i < L && (key & pmask) == prefix;
          const uint32_t bin = (key >> shift) & 0xffu;
          // the lanes that share the first active lane's bin add with one atomic
          const uint64_t act = __ballot(in);
          if (act != 0ull) {
            const int leader = __ffsll(static_cast<long long>(act)) - 1;
            const uint32_t lbin = static_cast<uint32_t>(__shfl(static_cast<int>(bin), leader));
            const uint64_t same = __ballot(in && bin == lbin);
            if (lane == leader) atomicAdd(&hist[lbin], static_cast<uint32_t>(__popcll(same)));
            if (in && bin != lbin) atomicAdd(&hist[bin], 1u);
          }
        }
      }
      __syncthreads();
      if (wave == 0) {
        // lane covers bins 255-4*lane down to 252-4*lane; lane 0 holds the top bins
        uint32_t c[4];
        uint32_t tot = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          c[j] = hist[255 - 4 * lane - j];
          tot += c[j];
        }
        uint32_t incl = tot;  // inclusive scan from lane 0
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const uint32_t v = __shfl_up(incl, o);
          if (lane >= o) incl += v;
        }
        const uint64_t hit = __ballot(incl >= kk);
        const int first = __ffsll(static_cast<long long>(hit)) - 1;  // kk <= matching count
        if (lane == first) {
          uint32_t above = incl - tot;
          int digit = 255 - 4 * lane;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (above + c[j] >= kk) {
              digit = 255 - 4 * lane - j;
              break;
            }
            above += c[j];
          }
          sh_digit = static_cast<uint32_t>(digit);
          sh_above = above;
        }
      }
      __syncthreads();
      prefix |= sh_digit << shift;
      pmask |= 0xffu << shift;
      kk -= sh_above;
      __syncthreads();  // hist and sh_* are rewritten by the next pass
    }
    thr = prefix;
    need_eq = kk;
    take_eq = true;
  }

  // (2) stable compaction in index order, in chunks of CH rounds.  Round r,
  //     wave w holds the indices r * 1024 + 64 w + lane, so the (r, w) pairs
  //     taken round-major are in index order.  Per chunk:
  //   a. every wave counts its keys above (gt) and equal to (eq) the
  //      threshold key in each round;
  //   b. one thread per (r, w): an exclusive scan of the eq counts gives the
  //      rank of the pair's first equal key; the equal keys taken are those
  //      ranked below need_eq, so the pair takes gt + clamp(need_eq - rank,
  //      0, eq) keys; an exclusive scan of those gives its first output slot;
  //   c. every lane writes its mask byte and, if taken, its index.
  //   A handful of barriers per chunk instead of three per round.
  constexpr int CH = kSelThreads / kSelWaves;  // 64 rounds: one (r, w) pair per thread in b
  __shared__ uint32_t c_eq[CH * kSelWaves], c_sel[CH * kSelWaves];
  __shared__ uint32_t s_tot[kSelWaves];
  auto for_rounds = [&](int r0, auto&& body) __attribute__((always_inline)) {
    if constexpr (R > 0) {
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (r >= r0 && r < r0 + CH) body(r, kr[r]);
    } else {
      const int r1 = r0 + CH < nr ? r0 + CH : nr;
      for (int r = r0; r < r1; ++r) body(r, key_of(r, r * kSelThreads + tid));
    }
  };
  auto scan_excl = [&](uint32_t v, uint32_t& total) __attribute__((always_inline)) -> uint32_t {
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t t = __shfl_up(incl, o);
      if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) s_tot[wave] = incl;
    __syncthreads();
    uint32_t before = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const uint32_t t = s_tot[w];
      before += w < wave ? t : 0u;
      total += t;
    }
    __syncthreads();  // s_tot is rewritten by the next scan
    return before + incl - v;
  };
  uint32_t base_eq = 0, base_sel = 0;
  for (int r0 = 0; r0 < nr; r0 += CH) {
    for_rounds(r0, [&](int r, uint32_t key) __attribute__((always_inline)) {
      const int i = r * kSelThreads + tid;
      const bool valid = i < L;
      const uint64_t bgt = __ballot(valid && key > thr);
      const uint64_t beq = __ballot(valid && take_eq && key == thr);
      if (lane == 0) {
        c_eq[(r - r0) * kSelWaves + wave] = static_cast<uint32_t>(__popcll(beq));
        c_sel[(r - r0) * kSelWaves + wave] = static_cast<uint32_t>(__popcll(bgt));
      }
    });
    __syncthreads();
    const bool ent = r0 + tid / kSelWaves < nr;  // this thread's pair exists
    const uint32_t veq = ent ? c_eq[tid] : 0u, vgt = ent ? c_sel[tid] : 0u;
    uint32_t tot_eq, tot_sel;
    const uint32_t rank = base_eq + scan_excl(veq, tot_eq);
    const uint32_t take = need_eq > rank ? (need_eq - rank < veq ? need_eq - rank : veq) : 0u;
    const uint32_t first = base_sel + scan_excl(vgt + take, tot_sel);
    c_eq[tid] = rank;
    c_sel[tid] = first;
    base_eq += tot_eq;
    base_sel += tot_sel;
    __syncthreads();
    for_rounds(r0, [&](int r, uint32_t key) __attribute__((always_inline)) {
      const int i = r * kSelThreads + tid;
      const bool valid = i < L;
      const bool gt = valid && key > thr;
      const bool eq = valid && take_eq && key == thr;
      const uint64_t beq = __ballot(eq);
      const uint32_t eq_before = c_eq[(r - r0) * kSelWaves + wave] + static_cast<uint32_t>(__popcll(beq & lt_mask));
      const bool sel = gt || (eq && eq_before < need_eq);
      const uint64_t bsel = __ballot(sel);
      const uint32_t pos = c_sel[(r - r0) * kSelWaves + wave] + static_cast<uint32_t>(__popcll(bsel & lt_mask));
      if (valid) {
        mask[i] = sel ? 1 : 0;
        if (sel) idx[pos] = idx_base + i;
      }
    });
    __syncthreads();  // c_eq / c_sel are rewritten by the next chunk
  }
  if (tid == 0 && n_sel != nullptr) *n_sel = static_cast<int32_t>(base_sel);
}

// Workgroup 0 selects; workgroup 1 (launched only when step_delta is not
// null) computes the step-level sum, independently of the selection.
template <int R>
__global__ void __launch_bounds__(kSelThreads)
select_rows(const float* __restrict__ s, int L, int k, int threshold_mode, float threshold,
            int32_t* __restrict__ idx, uint8_t* __restrict__ mask, int32_t* __restrict__ n_sel,
            const double* __restrict__ num, const double* __restrict__ den, double xi,
            double* __restrict__ step_delta) {
  if (blockIdx.x == 1) {
    step_delta_block(num, den, L, xi, step_delta);
    return;
  }
  topk_rows<R>(s, L, k, threshold_mode, threshold, 0, idx, mask, n_sel);
}

// Two-stage selection: workgroup t handles segment t (tokens [tN, tN + N)).
// A segment outside the anchor set clears its mask; an anchor segment takes
// its min(k, N) tokens ranked first by (s desc, index asc) and writes them at
// idx[a * min(k, N)...], a = the number of anchor segments before it, so idx
// stays ascending.  Workgroup 0 writes the total count.
template <int R>
__global__ void __launch_bounds__(kSelThreads)
select_segments(const float* __restrict__ s, const uint8_t* __restrict__ anchors, int T, int N, int k,
                int32_t* __restrict__ idx, uint8_t* __restrict__ mask, int32_t* __restrict__ n_sel) {
  __shared__ int sh_before, sh_total;
  const int t = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) {
    sh_before = 0;
    sh_total = 0;
  }
  __syncthreads();
  int before = 0, total = 0;
  for (int u = tid; u < T; u += kSelThreads) {
    const int a = anchors[u] != 0;
    total += a;
    before += (u < t) ? a : 0;
  }
  if (total) atomicAdd(&sh_total, total);
  if (before) atomicAdd(&sh_before, before);
  __syncthreads();
  const int kk = k < N ? k : N;
  if (t == 0 && tid == 0) *n_sel = sh_total * kk;
  const int64_t base = static_cast<int64_t>(t) * N;
  if (!anchors[t]) {
    for (int i = tid; i < N; i += kSelThreads) mask[base + i] = 0;
    return;
  }
  topk_rows<R>(s + base, N, kk, 0, 0.0f, static_cast<int>(base), idx + static_cast<int64_t>(sh_before) * kk,
               mask + base, nullptr);
}

// Anchor segments, one workgroup, T <= kMaxAnchorT:
//   mode 0: the k segments ranked first by (key desc, index asc), NaN first
//           (each segment counts the segments that rank before it);
//   mode 1: the evenly spaced segments floor((2j + 1) T / (2k)), j < k
//           (segment t is one iff some j satisfies 2kt <= (2j + 1) T < 2k(t + 1)).
constexpr int kMaxAnchorT = 4096;

__global__ void __launch_bounds__(kSelThreads)
anchor_select(const float* __restrict__ keys, int T, int k, int mode, uint8_t* __restrict__ anchors) {
  __shared__ uint32_t kl[kMaxAnchorT];
  const int tid = threadIdx.x;
  if (mode == 0) {
    for (int t = tid; t < T; t += kSelThreads) kl[t] = rank_key(keys[t]);
    __syncthreads();
    for (int t = tid; t < T; t += kSelThreads) {
      const uint32_t kt = kl[t];
      int rank = 0;
      for (int u = 0; u < T; ++u) {
        const uint32_t ku = kl[u];
        rank += (ku > kt || (ku == kt && u < t)) ? 1 : 0;
      }
      anchors[t] = rank < k ? 1 : 0;
    }
    return;
  }
  for (int t = tid; t < T; t += kSelThreads) {
    uint8_t a = 0;
    if (k > 0) {
      // smallest j with (2j + 1) T >= 2kt
      const int64_t num = 2 * static_cast<int64_t>(k) * t - T;
      const int64_t j = num <= 0 ? 0 : (num + 2 * static_cast<int64_t>(T) - 1) / (2 * static_cast<int64_t>(T));
      a = (j < k && (2 * j + 1) * T < 2 * static_cast<int64_t>(k) * (t + 1)) ? 1 : 0;
    }
    anchors[t] = a;
  }
}

hipError_t launch_saliency(int dtype_bf16, const void* x, const void* xref, const float* fw, int L, int N,
                           int D, double xi, float* s, double* num, double* den, double* step_delta,
                           hipStream_t stream) {
  const dim3 grid((L + (kSalThreads / kWave) - 1) / (kSalThreads / kWave));
  const int per_lane = (D / 8 + kWave - 1) / kWave;
  hipError_t e = hipErrorInvalidValue;
  bool done = false;
#define ECHO_SAL_CASE(MC)                                                                        \
  if (!done && (MC == 0 || per_lane <= MC)) {                                                    \
    done = true;                                                                                 \
    if (dtype_bf16)                                                                              \
      e = ECHO_LAUNCH("saliency_rows_bf16", (saliency_rows<bf16_t, MC>), grid, dim3(kSalThreads), \
                      0, stream, static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(xref), \
                      fw, L, N, D, xi, s, num, den);                                             \
    else                                                                                         \
      e = ECHO_LAUNCH("saliency_rows_f32", (saliency_rows<float, MC>), grid, dim3(kSalThreads),   \
                      0, stream, static_cast<const float*>(x), static_cast<const float*>(xref),   \
                      fw, L, N, D, xi, s, num, den);                                             \
  }
  ECHO_SAL_CASE(1)
  ECHO_SAL_CASE(2)
  ECHO_SAL_CASE(3)
  ECHO_SAL_CASE(4)
  ECHO_SAL_CASE(6)
  ECHO_SAL_CASE(8)
  ECHO_SAL_CASE(10)
  ECHO_SAL_CASE(12)
  ECHO_SAL_CASE(16)
  ECHO_SAL_CASE(0)
#undef ECHO_SAL_CASE
  if (e != hipSuccess || step_delta == nullptr) return e;
  return ECHO_LAUNCH("step_delta_sum", step_delta_sum, dim3(1), dim3(kSelThreads), 0, stream, num, den, L,
                     xi, step_delta);
}

hipError_t launch_topk(const float* s, int L, int k, int threshold_mode, float threshold, int32_t* idx,
                       uint8_t* mask, int32_t* n_sel, hipStream_t stream, const double* num,
                       const double* den, double xi, double* step_delta) {
  const dim3 grid(step_delta != nullptr ? 2 : 1);
#define ECHO_SEL_CASE(RK)                                                                      \
  if (L <= RK * kSelThreads)                                                                   \
    return ECHO_LAUNCH("select_rows", select_rows<RK>, grid, dim3(kSelThreads), 0, stream, s, L, \
                       k, threshold_mode, threshold, idx, mask, n_sel, num, den, xi, step_delta);
  ECHO_SEL_CASE(8)
  ECHO_SEL_CASE(32)
  ECHO_SEL_CASE(80)
#undef ECHO_SEL_CASE
  return ECHO_LAUNCH("select_rows", select_rows<0>, grid, dim3(kSelThreads), 0, stream, s, L, k,
                     threshold_mode, threshold, idx, mask, n_sel, num, den, xi, step_delta);
}

hipError_t launch_topk_segments(const float* s, const uint8_t* anchors, int T, int N, int k, int32_t* idx,
                                uint8_t* mask, int32_t* n_sel, hipStream_t stream) {
#define ECHO_SEG_CASE(RK)                                                                             \
  if (N <= RK * kSelThreads)                                                                          \
    return ECHO_LAUNCH("select_segments", select_segments<RK>, dim3(T), dim3(kSelThreads), 0, stream, s, \
                       anchors, T, N, k, idx, mask, n_sel);
  ECHO_SEG_CASE(2)
  ECHO_SEG_CASE(8)
  ECHO_SEG_CASE(32)
#undef ECHO_SEG_CASE
  return ECHO_LAUNCH("select_segments", select_segments<0>, dim3(T), dim3(kSelThreads), 0, stream, s, anchors,
                     T, N, k, idx, mask, n_sel);
}

int max_anchor_segments() { return kMaxAnchorT; }

hipError_t launch_anchors(const float* keys, int T, int k, int mode, uint8_t* anchors, hipStream_t stream) {
  return ECHO_LAUNCH("anchor_select", anchor_select, dim3(1), dim3(kSelThreads), 0, stream, keys, T, k, mode,
                     anchors);
}

hipError_t launch_select(int dtype_bf16, const void* x, const void* xref, const float* fw, int L, int N,
                         int D, double xi, int k, int threshold_mode, float threshold, float* s,
                         double* num, double* den, int32_t* idx, uint8_t* mask, int32_t* n_sel,
                         double* step_delta, hipStream_t stream) {
  // the step-level sum runs beside the selection, in the same launch
  const hipError_t e = launch_saliency(dtype_bf16, x, xref, fw, L, N, D, xi, s, num, den, nullptr, stream);
  if (e != hipSuccess) return e;
  return launch_topk(s, L, k, threshold_mode, threshold, idx, mask, n_sel, stream, num, den, xi, step_delta);
}

}  // namespace echo

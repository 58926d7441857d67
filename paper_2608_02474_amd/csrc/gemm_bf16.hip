// bf16 MFMA GEMM with fused epilogues for the projections of the partial DiT
// block (Sec. 3.3: Q for the active tokens, K/V for all tokens, output
// projection and FFN for the active tokens).
//
//   C[m, n] = epilogue( sum_k A[row(m), k] * B[n, k] + bias[n] )
//
// A is [M][K] row-major (optionally gathered through a row-index list, so the
// query projection reads the selected rows of the LN output in place); B is
// [N][K] row-major (nn.Linear weight layout), optionally split at n_split
// between two matrices so that K and V projections run as one N = 2D GEMM.
// Both operands are K-contiguous, which is what the MFMA operand layout wants:
// every lane feeds 8 consecutive k values (16 bytes).
//
// Tiling for gfx950: a BM x BN output tile per workgroup of WM x WN waves,
// each wave (BM/WM) x (BN/WN) as 32x32 blocks of v_mfma_f32_32x32x16_bf16.
// The build uses 256 x 256 tiles, 2 x 4 waves and a k-step of 32.  A and B
// tiles are copied straight from global memory into an NS-stage LDS ring
// (4 stages) with direct global-to-LDS loads (no VGPR staging; each lane
// fetches the 16-byte piece whose swizzled slot is its lane slot), one
// barrier per k-step.  LDS rows are BK * 2 bytes; the 16-byte chunk of row r
// is XOR-swizzled (by (r >> 2) & 3 for 64-byte rows, (r >> 1) & 7 for
// 128-byte rows) so that the rows one LDS cycle reads hit distinct bank
// groups.
// Workgroup ids are remapped so that each XCD (blocks are dealt round-robin
// to the 8 XCDs) owns a contiguous run of tiles, then grouped 8 tile-rows at
// a time so a run shares A and B panels in its L2.
// Requires N % BN == 0, n_split % BN == 0, K % BK == 0 and byte offsets of
// A and B rows below 2^31; M is arbitrary (tail rows clamp their loads and
// skip their stores).
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

// LDS rows hold BK bf16 (BK/8 chunks of 16 B).  The chunk of row r is
// XOR-swizzled so that the 16 consecutive rows one LDS cycle serves (256
// bytes = 2 rows of 128 B, or 4 rows of 64 B) land in 16 distinct bank groups.
template <int BK>
__device__ __forceinline__ int gslot(int row, int chunk) {
  if (BK == 64) return chunk ^ ((row >> 1) & 7);
  return chunk ^ ((row >> 2) & 3);
}

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// GELU with the tanh approximation, using 0.5 z (1 + tanh u) = z / (1 + e^{-2u});
// the reciprocal is the hardware one (1 ulp), far below the bf16 rounding of
// the result.
__device__ __forceinline__ float gelu_tanh_fast(float z) {
  const float u = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z * __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * u));
}

// Grouped tile order: 8 tile-rows at a time, down the rows first, so that
// consecutive tiles share B panels and a run of them shares A panels in L2.
__host__ __device__ __forceinline__ void gemm_tile_of(int pid, int tm, int tn, int& tile_m, int& tile_n) {
  constexpr int GROUP = 8;
  const int group_size = GROUP * tn;
  const int first_m = (pid / group_size) * GROUP;
  const int gm = (tm - first_m) < GROUP ? (tm - first_m) : GROUP;
  tile_m = first_m + (pid % group_size) % gm;
  tile_n = (pid % group_size) / gm;
}

// Bias (and gate) of the 4 consecutive output columns col .. col+3.
template <int EPI>
__device__ __forceinline__ void gemm_col4(const GemmBf16Args& p, int col, float* bias, float* gate) {
  const bf16_t* bias_p = col < p.n_split ? p.bias0 + col : p.bias1 + (col - p.n_split);
  const uint2 bb = *reinterpret_cast<const uint2*>(bias_p);
  bias[0] = __uint_as_float(bb.x << 16);
  bias[1] = __uint_as_float(bb.x & 0xffff0000u);
  bias[2] = __uint_as_float(bb.y << 16);
  bias[3] = __uint_as_float(bb.y & 0xffff0000u);
  if (EPI == EPI_GATE_RES) {
    const float4 g = *reinterpret_cast<const float4*>(p.gate + col);
    gate[0] = g.x; gate[1] = g.y; gate[2] = g.z; gate[3] = g.w;
  }
}

// Residual of the 4 consecutive columns col .. col+3 of row `row` (gathered
// through res_rows if given), bf16 or fp32, as fp32.
__device__ __forceinline__ void gemm_res4(const GemmBf16Args& p, int row, int col, float* res) {
  const int64_t rr = p.res_rows ? p.res_rows[row] : row;
  if (p.res_bf16) {
    const uint2 rb = ldg8_nt(static_cast<const bf16_t*>(p.res) + rr * p.ldr + col);
    res[0] = __uint_as_float(rb.x << 16);
    res[1] = __uint_as_float(rb.x & 0xffff0000u);
    res[2] = __uint_as_float(rb.y << 16);
    res[3] = __uint_as_float(rb.y & 0xffff0000u);
  } else {
    const uint4 rf = ldg16_nt(static_cast<const float*>(p.res) + rr * p.ldr + col);
    res[0] = __uint_as_float(rf.x); res[1] = __uint_as_float(rf.y); res[2] = __uint_as_float(rf.z); res[3] = __uint_as_float(rf.w);
  }
}

// Output of 4 consecutive columns col .. col+3 of row `row` (acc4 = sums
// without bias; res = the residual of those columns for EPI_GATE_RES).  The
// fp32 gate + residual outputs and their residual reads are streams read or
// written once, so they use the non-temporal accesses (O projection
// 0.687 -> 0.653 ms, FFN down 1.657 -> 1.645 ms); the bf16 outputs are read
// by the next kernel and keep ordinary stores.
template <int EPI>
__device__ __forceinline__ void gemm_store4(const GemmBf16Args& p, int row, int col, const float* acc4,
                                            const float* bias, const float* gate, const float* res) {
  float v[4] = {acc4[0] + bias[0], acc4[1] + bias[1], acc4[2] + bias[2], acc4[3] + bias[3]};
  if (EPI == EPI_GATE_RES) {
    float4 o;
    o.x = res[0] + gate[0] * v[0];
    o.y = res[1] + gate[1] * v[1];
    o.z = res[2] + gate[2] * v[2];
    o.w = res[3] + gate[3] * v[3];
    stg16_nt(static_cast<float*>(p.C) + static_cast<int64_t>(row) * p.ldc + col, make_uint4(__float_as_uint(o.x), __float_as_uint(o.y), __float_as_uint(o.z), __float_as_uint(o.w)));
  } else {
    if (EPI == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = gelu_tanh_fast(v[e]);
    }
    uint2 o;
    o.x = pack_bf16x2(v[0], v[1]);
    o.y = pack_bf16x2(v[2], v[3]);
    *reinterpret_cast<uint2*>(static_cast<bf16_t*>(p.C) + static_cast<int64_t>(row) * p.ldc + col) = o;
  }
}

template <int BM, int BN, int WM, int WN, int NS, int BK>
struct GemmCfg {
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kTM = BM / WM / 32;                 // 32x32 blocks per wave (rows)
  static constexpr int kTN = BN / WN / 32;                 // (columns)
  static constexpr int kRowBytes = BK * 2;
  static constexpr int kRowsPerCopy = 1024 / kRowBytes;     // rows one 1 KB copy fills
  static constexpr int kStageBytes = (BM + BN) * kRowBytes;  // A + B tiles
  static constexpr int kCopies = (BM + BN) / kRowsPerCopy / kWaves;  // per wave per k-step
  static_assert(BK == 32 || BK == 64, "k-step of 32 or 64");
  static_assert((BM + BN) % (kRowsPerCopy * kWaves) == 0, "copies split evenly over the waves");
  static_assert(BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "wave tile of 32x32 blocks");
  static_assert(NS >= 2 && NS <= 5 && NS * kStageBytes <= 160 * 1024, "LDS ring fits");
};

template <int BM, int BN, int WM, int WN, int NS, int BK, int EPI>
__global__ void __launch_bounds__(WM * WN * 64, 1) gemm_bf16_nt(GemmBf16Args p) {
  typedef GemmCfg<BM, BN, WM, WN, NS, BK> C;
  constexpr int CPR = BK / 8;  // 16-byte chunks per row
  __shared__ __attribute__((aligned(1024))) char smem[NS * C::kStageBytes];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave, l32 = lane & 31, hi = lane >> 5;
  const int wm = wave / WN, wn = wave % WN;

  // ---- tile id.  Unsplit launches take tiles [tile_base, tile_base +
  // gridDim.x) of the grouped order, remapped so that each XCD works through a
  // contiguous run; split launches give workgroup g k-range g % nsplit of tile
  // tile_base + g / nsplit.
  const int tm = (p.M + BM - 1) / BM, tn = p.N / BN;
  const bool split_k = p.nsplit > 1;
  int pid, ksplit = 0;
  if (!split_k) {
    const int total = gridDim.x, g = blockIdx.x;
    const int q = total / 8, r = total % 8, xcd = g % 8, loc = g / 8;
    pid = p.tile_base + xcd * q + (xcd < r ? xcd : r) + loc;
  } else {
    pid = p.tile_base + blockIdx.x / p.nsplit;
    ksplit = blockIdx.x % p.nsplit;
  }
  int tile_m, tile_n;
  gemm_tile_of(pid, tm, tn, tile_m, tile_n);
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // ---- copy plan: copy c of this wave fills kRowsPerCopy tile rows (1 KB) of
  // A (rows < BM) or B; the lane lands in row kRowsPerCopy * idx + lane / CPR,
  // slot lane % CPR.  The lane keeps a 32-bit byte offset into its matrix; the
  // matrix base (advanced by one k-step per iteration) is wave-uniform.
  uint32_t voff[C::kCopies];
  bool is_a[C::kCopies];
  uint32_t dst[C::kCopies];
  const uint32_t lds0 = lds_offset(smem);
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const bf16_t* b_base = n0 < p.n_split ? p.B0 : p.B1;  // BN divides n_split
  const int n_off = n0 < p.n_split ? n0 : n0 - p.n_split;
#pragma unroll
  for (int c = 0; c < C::kCopies; ++c) {
    const int idx = wave_u + C::kWaves * c;  // 1 KB block index within the stage
    const int row = C::kRowsPerCopy * idx + lane / CPR;  // row of the (A ++ B) stage
    const int chunk = gslot<BK>(row, lane % CPR);       // logical chunk in this lane's slot
    is_a[c] = C::kRowsPerCopy * idx < BM;
    if (is_a[c]) {
      int m = m0 + row;
      m = m < p.M ? m : p.M - 1;
      const uint32_t ar = p.a_rows ? static_cast<uint32_t>(p.a_rows[m]) : static_cast<uint32_t>(m);
      voff[c] = (ar * static_cast<uint32_t>(p.lda) + chunk * 8) * 2u;
    } else {
      const uint32_t n = n_off + row - BM;
      voff[c] = (n * static_cast<uint32_t>(p.ldb) + chunk * 8) * 2u;
    }
    dst[c] = lds0 + idx * 1024;
  }
  auto issue = [&](int kt, int stage) __attribute__((always_inline)) {
    const bf16_t* sa = p.A + static_cast<int64_t>(kt) * BK;
    const bf16_t* sb = b_base + static_cast<int64_t>(kt) * BK;
#pragma unroll
    for (int c = 0; c < C::kCopies; ++c)
      lds_copy16_s(is_a[c] ? sa : sb, voff[c], dst[c] + stage * C::kStageBytes);
  };
  // refill source of the running k-step (set once per k-step)
  const bf16_t* fill_a = p.A;
  const bf16_t* fill_b = b_base;
  uint32_t fill_off = 0;
  auto issue_one = [&](int c) __attribute__((always_inline)) {
    lds_copy16_s(is_a[c] ? fill_a : fill_b, voff[c], dst[c] + fill_off);
  };

  // ---- fragment read offsets (bytes within a stage): k16-step s reads chunk 2s + hi
  constexpr int KS = BK / 16;  // k16-steps per k-step
  int a_rd[KS], b_rd[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int ra = wm * (BM / WM) + l32;  // + i * 32 rows: same swizzle, folded into the offset
    const int rb = BM + wn * (BN / WN) + l32;
    a_rd[s] = ra * C::kRowBytes + gslot<BK>(ra, 2 * s + hi) * 16;
    b_rd[s] = rb * C::kRowBytes + gslot<BK>(rb, 2 * s + hi) * 16;
  }

  f32x16 acc[C::kTM][C::kTN];
#pragma unroll
  for (int i = 0; i < C::kTM; ++i)
#pragma unroll
    for (int j = 0; j < C::kTN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Fragments of two k16-steps live at once: step s+1 is read from LDS while
  // the MFMAs of step s run.  sched_barrier pins that order (left alone, the
  // scheduler hoists every read of a k-step above its MFMAs and runs out of
  // registers).
  bf16x8 fa[2][C::kTM], fb[2][C::kTN];
  auto load = [&](auto set_c, int stage, int s) __attribute__((always_inline)) {
    constexpr int SET = decltype(set_c)::value;
    const char* base = smem + stage * C::kStageBytes;  // stage is wave-uniform, not unrolled
#pragma unroll
    for (int i = 0; i < C::kTM; ++i)
      fa[SET][i] = *reinterpret_cast<const bf16x8*>(base + a_rd[s] + i * 32 * C::kRowBytes);
#pragma unroll
    for (int j = 0; j < C::kTN; ++j)
      fb[SET][j] = *reinterpret_cast<const bf16x8*>(base + b_rd[s] + j * 32 * C::kRowBytes);
  };
  // MFMAs of one fragment set over accumulator rows [I0, I1), with the
  // refill copies [Q0, Q1) spread evenly between them (group G of a k-step
  // carries copies [G * kPerGroup, (G + 1) * kPerGroup)).
  constexpr int kPerGroup = (C::kCopies + KS - 1) / KS;
  auto mma = [&](auto set_c, auto i0_c, auto i1_c, auto g_c) __attribute__((always_inline)) {
    constexpr int SET = decltype(set_c)::value;
    constexpr int IA = decltype(i0_c)::value, IB = decltype(i1_c)::value, G = decltype(g_c)::value;
    constexpr int NM = (IB - IA) * C::kTN;
    constexpr int Q0 = G * kPerGroup < C::kCopies ? G * kPerGroup : C::kCopies;
    constexpr int Q1 = Q0 + kPerGroup < C::kCopies ? Q0 + kPerGroup : C::kCopies;
    constexpr int NQ = Q1 - Q0;
#pragma unroll
    for (int i = IA; i < IB; ++i)
#pragma unroll
      for (int j = 0; j < C::kTN; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[SET][i], fb[SET][j], acc[i][j], 0, 0, 0);
        if constexpr (NQ > 0) {
          const int t = (i - IA) * C::kTN + j;
#pragma unroll
          for (int q = 0; q < NQ; ++q)
            if (t == q * NM / NQ) issue_one(Q0 + q);
        }
      }
  };
  typedef std::integral_constant<int, 0> I0;
  typedef std::integral_constant<int, C::kTM / 2> IH;
  typedef std::integral_constant<int, C::kTM> IM;
  typedef std::integral_constant<int, (KS - 1) & 1> ILAST;

  // NS-stage ring: k-step kt reads stage kt % NS while kt+1 .. kt+NS-1 are
  // in flight.  The barrier of k-step kt sits inside its last MFMA group:
  // before it, every wave has issued all its reads of stage kt % NS (which
  // k-step kt+1 refills with kt+NS) and waited until at most its copies of
  // the newest NS-2 k-steps are outstanding, so after it stage (kt+1) % NS is
  // complete and its first fragments are read under the remaining MFMAs.
  const int nk_all = p.K / BK;
  const int kt0 = split_k ? ksplit * p.kps : 0;  // first k-step of this workgroup
  const int nk = split_k ? (nk_all - kt0 < p.kps ? nk_all - kt0 : p.kps) : nk_all;  // >= 1
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nk) issue(kt0 + s, s);
  // Waits allow the copies of the NS-2 k-steps issued after the one needed;
  // a range of fewer than NS-1 k-steps issued fewer, so it drains them all.
  const bool short_range = nk < NS - 1;
  auto wait_next = [&]() __attribute__((always_inline)) {
    if (short_range)
      __builtin_amdgcn_s_waitcnt(0);
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((NS - 2) * C::kCopies));
  };
  wait_next();  // k-step 0 complete
  __syncthreads();
  load(I0{}, 0, 0);
  int stage = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const int next = stage + 1 == NS ? 0 : stage + 1;
    const int fill = stage == 0 ? NS - 1 : stage - 1;
    // k-step kt + NS - 1 goes to the stage read at kt - 1; past the end the
    // last k-step is fetched again (in bounds, never read) so that every
    // k-step issues the same copies and the wait below is uniform.
    const int kf = kt0 + (kt + NS - 1 < nk ? kt + NS - 1 : nk - 1);
    fill_a = p.A + static_cast<int64_t>(kf) * BK;
    fill_b = b_base + static_cast<int64_t>(kf) * BK;
    fill_off = fill * C::kStageBytes;
    static_for<0, KS - 1>([&](auto s_c) __attribute__((always_inline)) {
      constexpr int S = decltype(s_c)::value;
      __builtin_amdgcn_sched_barrier(0);
      load(std::integral_constant<int, (S + 1) & 1>{}, stage, S + 1);
      mma(std::integral_constant<int, S & 1>{}, I0{}, IM{}, s_c);
    });
    __builtin_amdgcn_sched_barrier(0);
    mma(ILAST{}, I0{}, IH{}, std::integral_constant<int, KS - 1>{});
    __builtin_amdgcn_sched_barrier(0);
    wait_next();  // k-step kt+1 complete
    __syncthreads();
    if (kt + 1 < nk) load(I0{}, next, 0);
    mma(ILAST{}, IH{}, IM{}, std::integral_constant<int, KS>{});
    __builtin_amdgcn_sched_barrier(0);
    stage = next;
  }
  __builtin_amdgcn_s_waitcnt(0);  // refetched k-steps still landing in LDS

  // ---- epilogue.  The 32x32 accumulator layout (lane holds column l32 and
  // rows 8*(r/4) + 4*hi + r%4 of register r) is turned into row-contiguous
  // pieces through LDS: each wave stages one 32-row slab of its tile at a
  // time in a private region and reads it back as 4 consecutive columns per
  // lane, so bias, gate and residual are read and the output written 8-16
  // bytes per lane.  Staged rows are padded by 8 floats: the two half-waves
  // (rows r and r+4) then write disjoint bank halves.
  constexpr int WCOLS = C::kTN * 32;        // columns of a wave tile
  constexpr int EP_LD = WCOLS + 8;          // staged row stride (floats)
  constexpr int LPR = WCOLS / 4;            // lanes per staged row
  constexpr int RPI = kWave / LPR;          // rows per read instruction
  static_assert(C::kWaves * 32 * EP_LD * 4 <= NS * C::kStageBytes, "epilogue staging fits the ring");
  __syncthreads();  // every wave is done with the ring
  float* ep = reinterpret_cast<float*>(smem) + wave * 32 * EP_LD;
  const int c_l = (lane % LPR) * 4;                   // first of this lane's 4 columns
  const int col = n0 + wn * (BN / WN) + c_l;           // global column (4 | col)
  float bias[4], gate[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (!split_k) gemm_col4<EPI>(p, col, bias, gate);
  constexpr int NQ = 32 / RPI;                     // row groups of a slab per lane
  constexpr int NR = EPI == EPI_GATE_RES ? NQ : 1;
#pragma unroll
  for (int i = 0; i < C::kTM; ++i) {
    // the residuals of this lane's rows of the slab: every row index, then
    // every residual, loaded together (rows past M load row M - 1, unused),
    // in flight while the slab is staged
    float res[NR][4];
    if constexpr (EPI == EPI_GATE_RES) {
      if (!split_k) {
        int64_t rr[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int row = m0 + wm * (BM / WM) + i * 32 + q * RPI + lane / LPR;
          rr[q] = row < p.M ? row : p.M - 1;
        }
        if (p.res_rows != nullptr) {
          int g[NQ];
#pragma unroll
          for (int q = 0; q < NQ; ++q) g[q] = p.res_rows[rr[q]];
#pragma unroll
          for (int q = 0; q < NQ; ++q) rr[q] = g[q];
        }
        if (p.res_bf16) {
          const bf16_t* rb = static_cast<const bf16_t*>(p.res) + col;
          uint2 raw[NQ];
#pragma unroll
          for (int q = 0; q < NQ; ++q) raw[q] = ldg8_nt(rb + rr[q] * p.ldr);
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            res[q][0] = __uint_as_float(raw[q].x << 16);
            res[q][1] = __uint_as_float(raw[q].x & 0xffff0000u);
            res[q][2] = __uint_as_float(raw[q].y << 16);
            res[q][3] = __uint_as_float(raw[q].y & 0xffff0000u);
          }
        } else {
          const float* rf = static_cast<const float*>(p.res) + col;
          uint4 raw[NQ];
#pragma unroll
          for (int q = 0; q < NQ; ++q) raw[q] = ldg16_nt(rf + rr[q] * p.ldr);
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            res[q][0] = __uint_as_float(raw[q].x);
            res[q][1] = __uint_as_float(raw[q].y);
            res[q][2] = __uint_as_float(raw[q].z);
            res[q][3] = __uint_as_float(raw[q].w);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < C::kTN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        ep[(8 * (r >> 2) + 4 * hi + (r & 3)) * EP_LD + j * 32 + l32] = acc[i][j][r];
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(63));  // this wave's staged slab is in LDS (LDS only)
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int r_l = q * RPI + lane / LPR;
      const int trow = wm * (BM / WM) + i * 32 + r_l;  // row within the tile
      const float4 a4 = *reinterpret_cast<const float4*>(ep + r_l * EP_LD + c_l);
      if (split_k) {
        // raw partial sums of this k-range, tile-local [BM][BN] per workgroup
        *reinterpret_cast<float4*>(p.part + static_cast<int64_t>(blockIdx.x) * BM * BN +
                                   static_cast<int64_t>(trow) * BN + (col - n0)) = a4;
      } else if (m0 + trow < p.M) {
        const float v[4] = {a4.x, a4.y, a4.z, a4.w};
        gemm_store4<EPI>(p, m0 + trow, col, v, bias, gate, res[EPI == EPI_GATE_RES ? q : 0]);
      }
    }
  }
}

// Sum the k-range partials of the split tail tiles in split order and apply
// the epilogue.  One thread per 4 output columns.
template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(256) gemm_splitk_reduce(GemmBf16Args p, int ntail) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(ntail) * BM * (BN / 4)) return;
  const int c4 = static_cast<int>(e % (BN / 4)), trow = static_cast<int>((e / (BN / 4)) % BM);
  const int j = static_cast<int>(e / (static_cast<int64_t>(BM) * (BN / 4)));
  const int tm = (p.M + BM - 1) / BM, tn = p.N / BN;
  int tile_m, tile_n;
  gemm_tile_of(p.tile_base + j, tm, tn, tile_m, tile_n);
  const int row = tile_m * BM + trow;
  if (row >= p.M) return;
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int sp = 0; sp < p.nsplit; ++sp) {
    const float4 a4 = *reinterpret_cast<const float4*>(
        p.part + (static_cast<int64_t>(j) * p.nsplit + sp) * BM * BN + static_cast<int64_t>(trow) * BN + 4 * c4);
    v[0] += a4.x;
    v[1] += a4.y;
    v[2] += a4.z;
    v[3] += a4.w;
  }
  float bias[4], gate[4] = {0.0f, 0.0f, 0.0f, 0.0f}, res[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  gemm_col4<EPI>(p, tile_n * BN + 4 * c4, bias, gate);
  if (EPI == EPI_GATE_RES) gemm_res4(p, row, tile_n * BN + 4 * c4, res);
  gemm_store4<EPI>(p, row, tile_n * BN + 4 * c4, v, bias, gate, res);
}

template <int BM, int BN, int WM, int WN, int NS, int BK, int EPI>
hipError_t launch_gemm_epi(const char* name, GemmBf16Args a, hipStream_t stream) {
  typedef GemmCfg<BM, BN, WM, WN, NS, BK> C;
  const int tiles = ((a.M + BM - 1) / BM) * (a.N / BN);
  const int nk = a.K / BK;
  // Tiles beyond the last full round (one workgroup per CU) are split along
  // k so that together they fill that round; a reduce kernel adds the splits.
  const int ncu = device_cu_count();
  const int tail = tiles % ncu;
  int nsplit = tail > 0 ? ncu / tail : 1;
  nsplit = nsplit < nk ? nsplit : nk;
  // Each split also writes and the reduce reads a 256 KB fp32 partial tile:
  // below about 20 k-steps per split that costs more than the shorter range
  // saves (160 k-steps: 8 splits beat 16 by 7-11 us; 432: 16 beat 8).
  constexpr int kMinStepsPerSplit = 20;
  const int cap = nk / kMinStepsPerSplit > 1 ? nk / kMinStepsPerSplit : 1;
  nsplit = nsplit < cap ? nsplit : cap;
  const size_t unit_bytes = sizeof(float) * BM * BN;
  while (nsplit > 1 && static_cast<size_t>(tail) * nsplit * unit_bytes > a.part_bytes) --nsplit;
  if (a.part == nullptr) nsplit = 1;
  ::echo::TimedLaunch scope(name, stream);
  a.tile_base = 0;
  if (nsplit < 2) {
    a.nsplit = 1;
    hipLaunchKernelGGL((gemm_bf16_nt<BM, BN, WM, WN, NS, BK, EPI>), dim3(tiles), dim3(C::kThreads), 0, stream, a);
    return hipGetLastError();
  }
  a.kps = (nk + nsplit - 1) / nsplit;  // k-steps per split
  nsplit = (nk + a.kps - 1) / a.kps;   // every split non-empty
  const int full = tiles - tail;
  if (full > 0) {
    a.nsplit = 1;
    hipLaunchKernelGGL((gemm_bf16_nt<BM, BN, WM, WN, NS, BK, EPI>), dim3(full), dim3(C::kThreads), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  a.tile_base = full;
  a.nsplit = nsplit;
  hipLaunchKernelGGL((gemm_bf16_nt<BM, BN, WM, WN, NS, BK, EPI>), dim3(tail * nsplit), dim3(C::kThreads), 0,
                     stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t threads = static_cast<int64_t>(tail) * BM * (BN / 4);
  hipLaunchKernelGGL((gemm_splitk_reduce<BM, BN, EPI>), dim3(static_cast<unsigned>((threads + 255) / 256)),
                     dim3(256), 0, stream, a, tail);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int NS, int BK>
hipError_t launch_gemm_tile(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream) {
  if (a.N % BN != 0 || (a.n_split < a.N && a.n_split % BN != 0) || a.K % BK != 0)
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_BIAS: return launch_gemm_epi<BM, BN, WM, WN, NS, BK, EPI_BIAS>(name, a, stream);
    case EPI_GELU: return launch_gemm_epi<BM, BN, WM, WN, NS, BK, EPI_GELU>(name, a, stream);
    default: return launch_gemm_epi<BM, BN, WM, WN, NS, BK, EPI_GATE_RES>(name, a, stream);
  }
}

hipError_t launch_gemm_bf16(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream) {
  if (a.M <= 0) return hipSuccess;
  // the tile loads address A and B through 32-bit byte offsets
  const int64_t lim = int64_t(1) << 31;
  if (a.a_nrows <= 0 || a.a_nrows * a.lda * 2 >= lim || int64_t(a.N) * a.ldb * 2 >= lim)
    return hipErrorInvalidValue;
  return launch_gemm_tile<256, 256, 2, 4, 4, 32>(name, epi, a, stream);
}

}  // namespace echo

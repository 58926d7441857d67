// The Wan-style block extras on the restricted-query path: qk RMSNorm with 3D
// rotary position embedding, applied in place to the q and k projections, the
// rotary angle table it reads, and a small vector kernel for the constant
// operands of the cross-attention sub-layer.
//
// qk_norm_rope_rows: one wave per row, the row held in registers as raw
//   16-byte vectors (all loads issued before the first is used); the RMSNorm
//   weight and the angle table staged once per workgroup in LDS, each wave
//   looping over rows.  The sum of
//   squares is reduced in fp32; every element is scaled by 1 / sqrt(ss / D +
//   eps) and the RMSNorm weight, then each channel pair (2j, 2j + 1) of a head
//   is rotated by the angle of its axis: the first nt pairs by the token's
//   frame t, the next nr by its grid row r, the last nc by its grid column c.
//   An 8-element chunk holds four whole pairs, so a lane rotates its own data.
// rope_table: (cos, sin) of p * base^(-j / n) for every axis position p and
//   pair j < n of the axis, computed in fp64 and stored as fp32 pairs.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kWanThreads = 256;
constexpr int kWanWaves = kWanThreads / kWave;

void rope_split(int dh, int* nt, int* nr, int* nc) {
  *nr = dh / 6;
  *nc = dh / 6;
  *nt = dh / 2 - 2 * (dh / 6);
}

int rope_table_entries(int T, int gh, int gw, int dh) {
  int nt, nr, nc;
  rope_split(dh, &nt, &nr, &nc);
  return T * nt + gh * nr + gw * nc;
}

__global__ void __launch_bounds__(256)
rope_table(int T, int gh, int gw, int nt, int nr, int nc, double base, float2* __restrict__ tab) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int e_t = T * nt, e_r = gh * nr, e_c = gw * nc;
  if (i >= e_t + e_r + e_c) return;
  int p, j, n;
  if (i < e_t) {
    p = i / nt, j = i % nt, n = nt;
  } else if (i < e_t + e_r) {
    p = (i - e_t) / nr, j = (i - e_t) % nr, n = nr;
  } else {
    p = (i - e_t - e_r) / nc, j = (i - e_t - e_r) % nc, n = nc;
  }
  const double ang = static_cast<double>(p) * pow(base, -static_cast<double>(j) / static_cast<double>(n));
  double s, c;
  sincos(ang, &s, &c);
  tab[i] = make_float2(static_cast<float>(c), static_cast<float>(s));
}

struct RopeGeom {
  const float2* tab;  // nullptr: RMSNorm only
  int L, gh, gw, T;   // token index = row % L (rows of a batch are b * L + i)
  int nt, nr, nc, dh;
};

// MAXC > 0: the row stays in registers (D <= 512 MAXC); MAXC == 0 reads it twice.
// STAGE: the workgroup first copies the RMSNorm weight and the angle table to
// LDS and each wave then loops over rows (row = 4 blockIdx.x + wave, in steps
// of 4 gridDim.x): read from L2 for every row, the weight (fp32) and the
// table entries moved four times the row's own bytes through the load path.
// SAME: a lane's chunks, 512 elements apart, hold the same pairs of their
// heads (the head size divides 512), so the four angles are read once a row.
template <int MAXC, bool STAGE, bool SAME = false>
__global__ void __launch_bounds__(kWanThreads)
qk_norm_rope_rows(bf16_t* __restrict__ z, int64_t ldz, int M, int D, const float* __restrict__ g, float eps,
                  const int32_t* __restrict__ rows, RopeGeom geo) {
  extern __shared__ float4 qkn_lds[];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int off_r = geo.T * geo.nt, off_c = off_r + geo.gh * geo.nr;  // first entries of the row and column axes
  float* gl = reinterpret_cast<float*>(qkn_lds);                     // [D] weight (STAGE)
  float2* tl = reinterpret_cast<float2*>(gl + D);                    // [off_c + gw nc] table (STAGE)
  if constexpr (STAGE) {
    const int ntab = geo.tab != nullptr ? off_c + geo.gw * geo.nc : 0;
    for (int i = threadIdx.x; i < D / 4; i += kWanThreads)
      reinterpret_cast<float4*>(gl)[i] = reinterpret_cast<const float4*>(g)[i];
    for (int i = threadIdx.x; i < ntab; i += kWanThreads) tl[i] = geo.tab[i];
    __syncthreads();
  }
  const int nch = D / 8;
  auto inv_rms = [&](float ss) __attribute__((always_inline)) {
    return __frcp_rn(__fsqrt_rn(__fadd_rn(__fdiv_rn(ss, static_cast<float>(D)), eps)));
  };
  const int64_t step = STAGE ? static_cast<int64_t>(gridDim.x) * kWanWaves : static_cast<int64_t>(M);
  for (int64_t m = static_cast<int64_t>(blockIdx.x) * kWanWaves + wave; m < M; m += step) {
    bf16_t* zr = z + m * ldz;
    int t = 0, r = 0, c = 0;
    if (geo.tab != nullptr) {
      const int tok = static_cast<int>((rows != nullptr ? static_cast<int64_t>(rows[m]) : m) % geo.L);
      t = tok / (geo.gh * geo.gw);
      r = (tok / geo.gw) % geo.gh;
      c = tok % geo.gw;
    }
    // (cos, sin) of pair jp of this row's token: the entry of the pair's axis,
    // chosen without a branch (lanes of a wave hold pairs of different axes)
    auto angle = [&](int jp) __attribute__((always_inline)) {
      const int it = t * geo.nt + jp;
      const int ir = off_r + r * geo.nr + (jp - geo.nt);
      const int ic = off_c + c * geo.nc + (jp - geo.nt - geo.nr);
      const int e = jp < geo.nt ? it : (jp < geo.nt + geo.nr ? ir : ic);
      return STAGE ? tl[e] : geo.tab[e];
    };
    // A lane's chunks lie 512 elements apart; when the head size divides 512
    // they all hold the same four pairs of their heads, whose angles are then
    // read once per row.
    constexpr bool same_pairs = SAME;  // set by the launcher when dh divides 512 or there is no table
    float2 cs_row[4];
    if constexpr (same_pairs) {
      if (geo.tab != nullptr) {
        const int p0 = ((lane * 8) % geo.dh) / 2;
#pragma unroll
        for (int q = 0; q < 4; ++q) cs_row[q] = angle(p0 + q);
      }
    }
    // normalise, weight and rotate the 8 elements of chunk ch in place
    auto finish = [&](float* v, int ch, float inv) __attribute__((always_inline)) {
      float gv[8];
      if constexpr (STAGE) {
        const float4 g0 = reinterpret_cast<const float4*>(gl + ch * 8)[0];
        const float4 g1 = reinterpret_cast<const float4*>(gl + ch * 8)[1];
        gv[0] = g0.x; gv[1] = g0.y; gv[2] = g0.z; gv[3] = g0.w;
        gv[4] = g1.x; gv[5] = g1.y; gv[6] = g1.z; gv[7] = g1.w;
      } else {
        unpack16(ldg16(g + ch * 8), gv, static_cast<const float*>(nullptr));
        unpack16(ldg16(g + ch * 8 + 4), gv + 4, static_cast<const float*>(nullptr));
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = __fmul_rn(__fmul_rn(v[j], inv), gv[j]);
      if (geo.tab == nullptr) return;
      const int p0 = ((ch * 8) % geo.dh) / 2;  // pair index of the chunk's first pair within its head
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float2 cs;
        if constexpr (same_pairs)
          cs = cs_row[q];
        else
          cs = angle(p0 + q);
        const float a = v[2 * q], b = v[2 * q + 1];
        v[2 * q] = __fsub_rn(__fmul_rn(a, cs.x), __fmul_rn(b, cs.y));
        v[2 * q + 1] = __fadd_rn(__fmul_rn(a, cs.y), __fmul_rn(b, cs.x));
      }
    };
    if constexpr (MAXC > 0) {
      Raw8<bf16_t> raw[MAXC];
#pragma unroll
      for (int u = 0; u < MAXC; ++u) {
        const int ch = lane + u * kWave;
        raw[u].load(zr + (ch < nch ? ch : nch - 1) * 8);
      }
      float ss = 0.0f;
#pragma unroll
      for (int u = 0; u < MAXC; ++u) {
        float v[8];
        raw[u].unpack(v);
        const bool ok = lane + u * kWave < nch;
#pragma unroll
        for (int j = 0; j < 8; ++j) ss += ok ? v[j] * v[j] : 0.0f;
      }
      const float inv = inv_rms(wave_sum(ss));
      // unpack again below rather than keep the first pass's floats live
      // (twice the row's registers)
#pragma unroll
      for (int u = 0; u < MAXC; ++u)
        asm volatile("" : "+v"(raw[u].v.x), "+v"(raw[u].v.y), "+v"(raw[u].v.z), "+v"(raw[u].v.w));
#pragma unroll
      for (int u = 0; u < MAXC; ++u) {
        const int ch = lane + u * kWave;
        if (ch < nch) {
          float v[8];
          raw[u].unpack(v);
          finish(v, ch, inv);
          stg16(zr + ch * 8, pack16(v, static_cast<const bf16_t*>(nullptr)));
        }
        // one chunk at a time: hoisting every chunk's weight and table reads
        // ahead of the first store doubled the registers and halved the waves
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      float ss = 0.0f;
      for (int ch = lane; ch < nch; ch += kWave) {
        float v[8];
        unpack16(ldg16(zr + ch * 8), v, static_cast<const bf16_t*>(nullptr));
#pragma unroll
        for (int j = 0; j < 8; ++j) ss += v[j] * v[j];
      }
      const float inv = inv_rms(wave_sum(ss));
      for (int ch = lane; ch < nch; ch += kWave) {
        float v[8];
        unpack16(ldg16(zr + ch * 8), v, static_cast<const bf16_t*>(nullptr));
        finish(v, ch, inv);
        stg16(zr + ch * 8, pack16(v, static_cast<const bf16_t*>(nullptr)));
      }
    }
  }
}

// out[i] = (a ? a[i] : 0) + beta
__global__ void __launch_bounds__(256)
vec_shift(const float* __restrict__ a, float beta, float* __restrict__ out, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = (a != nullptr ? a[i] : 0.0f) + beta;
}

hipError_t launch_rope_table(int T, int gh, int gw, int dh, double base, float2* tab, hipStream_t stream) {
  int nt, nr, nc;
  rope_split(dh, &nt, &nr, &nc);
  const int n = T * nt + gh * nr + gw * nc;
  return ECHO_LAUNCH("rope_table", rope_table, dim3((n + 255) / 256), dim3(256), 0, stream, T, gh, gw, nt, nr, nc,
                     base, tab);
}

hipError_t launch_qk_norm_rope(bf16_t* z, int64_t ldz, int M, int D, const float* g, float eps,
                               const int32_t* rows, const float2* tab, int L, int T, int gh, int gw, int dh,
                               hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  RopeGeom geo{tab, L, gh, gw, T, 0, 0, 0, dh};
  rope_split(dh, &geo.nt, &geo.nr, &geo.nc);
  const dim3 grid(static_cast<unsigned>((M + kWanWaves - 1) / kWanWaves));
  const int per_lane = (D / 8 + kWave - 1) / kWave;
  // weight and table in LDS when they fit four workgroups per CU
  const size_t ntab = tab != nullptr ? size_t(T) * geo.nt + size_t(gh) * geo.nr + size_t(gw) * geo.nc : 0;
  const size_t lds = sizeof(float) * size_t(D) + sizeof(float2) * ntab;
  if (lds <= 40960) {
    const unsigned cap = 4u * static_cast<unsigned>(device_cu_count());
    const dim3 grid_s(grid.x < cap ? grid.x : cap);
#define ECHO_QKS_CASE(MC)                                                                                      \
  if (per_lane <= MC) {                                                                                        \
    if (tab == nullptr || 512 % dh == 0)                                                                       \
      return ECHO_LAUNCH("qk_norm_rope", (qk_norm_rope_rows<MC, true, true>), grid_s, dim3(kWanThreads), lds,   \
                         stream, z, ldz, M, D, g, eps, rows, geo);                                            \
    return ECHO_LAUNCH("qk_norm_rope", (qk_norm_rope_rows<MC, true, false>), grid_s, dim3(kWanThreads), lds,    \
                       stream, z, ldz, M, D, g, eps, rows, geo);                                              \
  }
    ECHO_QKS_CASE(1)
    ECHO_QKS_CASE(2)
    ECHO_QKS_CASE(4)
    ECHO_QKS_CASE(8)
    ECHO_QKS_CASE(10)
    ECHO_QKS_CASE(16)
#undef ECHO_QKS_CASE
  }
#define ECHO_QKN_CASE(MC)                                                                                   \
  if (per_lane <= MC)                                                                                       \
    return ECHO_LAUNCH("qk_norm_rope", (qk_norm_rope_rows<MC, false>), grid, dim3(kWanThreads), 0, stream, z, ldz, \
                       M, D, g, eps, rows, geo);
  ECHO_QKN_CASE(1)
  ECHO_QKN_CASE(2)
  ECHO_QKN_CASE(4)
  ECHO_QKN_CASE(8)
  ECHO_QKN_CASE(10)
  ECHO_QKN_CASE(16)
#undef ECHO_QKN_CASE
  return ECHO_LAUNCH("qk_norm_rope", (qk_norm_rope_rows<0, false>), grid, dim3(kWanThreads), 0, stream, z, ldz, M,
                     D, g, eps, rows, geo);
}

hipError_t launch_vec_shift(const float* a, float beta, float* out, int n, hipStream_t stream) {
  return ECHO_LAUNCH("vec_shift", vec_shift, dim3((n + 255) / 256), dim3(256), 0, stream, a, beta, out, n);
}

}  // namespace echo

// The Wan-style block extras on the restricted-query path: qk RMSNorm with 3D
// rotary position embedding, applied in place to the q and k projections, the
// rotary angle table it reads, and a small vector kernel for the constant
// operands of the cross-attention sub-layer.
//
// qk_norm_rope_rows: one wave per row, the row held in registers as raw
//   16-byte vectors (all loads issued before the first is used).  The sum of
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
template <int MAXC>
__global__ void __launch_bounds__(kWanThreads)
qk_norm_rope_rows(bf16_t* __restrict__ z, int64_t ldz, int M, int D, const float* __restrict__ g, float eps,
                  const int32_t* __restrict__ rows, RopeGeom geo) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t m = static_cast<int64_t>(blockIdx.x) * kWanWaves + wave;
  if (m >= M) return;
  bf16_t* zr = z + m * ldz;
  const int nch = D / 8;
  int t = 0, r = 0, c = 0;
  if (geo.tab != nullptr) {
    const int tok = static_cast<int>((rows != nullptr ? static_cast<int64_t>(rows[m]) : m) % geo.L);
    t = tok / (geo.gh * geo.gw);
    r = (tok / geo.gw) % geo.gh;
    c = tok % geo.gw;
  }
  const float2* tab_t = geo.tab;
  const float2* tab_r = geo.tab + geo.T * geo.nt;
  const float2* tab_c = tab_r + geo.gh * geo.nr;
  // normalise, weight and rotate the 8 elements of chunk ch in place
  auto finish = [&](float* v, int ch, float inv) __attribute__((always_inline)) {
    float gv[8];
    unpack16(ldg16(g + ch * 8), gv, static_cast<const float*>(nullptr));
    unpack16(ldg16(g + ch * 8 + 4), gv + 4, static_cast<const float*>(nullptr));
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = __fmul_rn(__fmul_rn(v[j], inv), gv[j]);
    if (geo.tab == nullptr) return;
    const int p0 = ((ch * 8) % geo.dh) / 2;  // pair index of the chunk's first pair within its head
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int jp = p0 + q;
      // table entry of the pair's axis, chosen without a branch (lanes of a
      // wave hold pairs of different axes)
      const int it = t * geo.nt + jp;
      const int ir = (tab_r - tab_t) + r * geo.nr + (jp - geo.nt);
      const int ic = (tab_c - tab_t) + c * geo.nc + (jp - geo.nt - geo.nr);
      const int e = jp < geo.nt ? it : (jp < geo.nt + geo.nr ? ir : ic);
      const float2 cs = tab_t[e];
      const float a = v[2 * q], b = v[2 * q + 1];
      v[2 * q] = __fsub_rn(__fmul_rn(a, cs.x), __fmul_rn(b, cs.y));
      v[2 * q + 1] = __fadd_rn(__fmul_rn(a, cs.y), __fmul_rn(b, cs.x));
    }
  };
  auto inv_rms = [&](float ss) __attribute__((always_inline)) {
    return __frcp_rn(__fsqrt_rn(__fadd_rn(__fdiv_rn(ss, static_cast<float>(D)), eps)));
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
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
      const int ch = lane + u * kWave;
      if (ch < nch) {
        float v[8];
        raw[u].unpack(v);
        finish(v, ch, inv);
        stg16(zr + ch * 8, pack16(v, static_cast<const bf16_t*>(nullptr)));
      }
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
#define ECHO_QKN_CASE(MC)                                                                                   \
  if (per_lane <= MC)                                                                                       \
    return ECHO_LAUNCH("qk_norm_rope", qk_norm_rope_rows<MC>, grid, dim3(kWanThreads), 0, stream, z, ldz, M, D, \
                       g, eps, rows, geo);
  ECHO_QKN_CASE(1)
  ECHO_QKN_CASE(2)
  ECHO_QKN_CASE(4)
  ECHO_QKN_CASE(8)
  ECHO_QKN_CASE(10)
  ECHO_QKN_CASE(16)
#undef ECHO_QKN_CASE
  return ECHO_LAUNCH("qk_norm_rope", qk_norm_rope_rows<0>, grid, dim3(kWanThreads), 0, stream, z, ldz, M, D, g,
                     eps, rows, geo);
}

hipError_t launch_vec_shift(const float* a, float beta, float* out, int n, hipStream_t stream) {
  return ECHO_LAUNCH("vec_shift", vec_shift, dim3((n + 255) / 256), dim3(256), 0, stream, a, beta, out, n);
}

}  // namespace echo

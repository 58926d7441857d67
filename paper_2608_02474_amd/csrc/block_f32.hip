// fp32 path of the partial DiT block for small shapes (any head width up to
// 128): a plain LDS-tiled fp32 GEMM with the same fused epilogues as the bf16
// MFMA GEMM, and a one-wave-per-(query, head) streaming-softmax attention.
// These kernels exist for exactness checks at fp32 and are not tuned.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int F32_TILE = 16;

__device__ __forceinline__ float gelu_tanh_ref(float z) {
  return 0.5f * z * (1.0f + tanhf(0.7978845608028654f * (z + 0.044715f * z * z * z)));
}

template <int EPI>  // 0 bias, 1 gelu, 2 gate+residual (same codes as the bf16 GEMM)
__global__ void __launch_bounds__(F32_TILE * F32_TILE) gemm_f32_nt(GemmF32Args p) {
  __shared__ float As[F32_TILE][F32_TILE + 1];
  __shared__ float Bs[F32_TILE][F32_TILE + 1];
  const int tx = threadIdx.x % F32_TILE, ty = threadIdx.x / F32_TILE;
  const int row = blockIdx.y * F32_TILE + ty;
  const int col = blockIdx.x * F32_TILE + tx;
  const int arow_l = blockIdx.y * F32_TILE + ty;   // row this thread stages from A
  const int brow_l = blockIdx.x * F32_TILE + ty;   // row this thread stages from B
  const float* arow = nullptr;
  if (arow_l < p.M) arow = p.A + (p.a_rows ? static_cast<int64_t>(p.a_rows[arow_l]) : arow_l) * p.lda;
  const float* brow = nullptr;
  if (brow_l < p.N)
    brow = brow_l < p.n_split ? p.B0 + static_cast<int64_t>(brow_l) * p.ldb
                              : p.B1 + static_cast<int64_t>(brow_l - p.n_split) * p.ldb;
  float acc = 0.0f;
  for (int k0 = 0; k0 < p.K; k0 += F32_TILE) {
    const int kk = k0 + tx;
    As[ty][tx] = (arow && kk < p.K) ? arow[kk] : 0.0f;
    Bs[ty][tx] = (brow && kk < p.K) ? brow[kk] : 0.0f;
    __syncthreads();
#pragma unroll
    for (int t = 0; t < F32_TILE; ++t) acc += As[ty][t] * Bs[tx][t];
    __syncthreads();
  }
  if (row >= p.M || col >= p.N) return;
  const float v = acc + (col < p.n_split ? p.bias0[col] : p.bias1[col - p.n_split]);
  float outv;
  if (EPI == 0) {
    outv = v;
  } else if (EPI == 1) {
    outv = gelu_tanh_ref(v);
  } else {
    const int64_t rr = p.res_rows ? p.res_rows[row] : row;
    outv = p.res[rr * p.ldr + col] + p.gate[col] * v;
  }
  p.C[static_cast<int64_t>(row) * p.ldc + col] = outv;
}

// One wave per (query row, head); keys in chunks of 64 (one per lane).
__global__ void __launch_bounds__(kWave)
attn_fwd_f32(const float* __restrict__ q, int64_t ldq, const float* __restrict__ k,
             const float* __restrict__ v, int64_t ldkv, int Mq, int L, int dh, float scale,
             float* __restrict__ out, int64_t ldo) {
  __shared__ float qs[128];
  __shared__ float ps[kWave];
  const int lane = threadIdx.x;
  const int qr = blockIdx.x, head = blockIdx.y;
  const int64_t hoff = static_cast<int64_t>(head) * dh;
  for (int d = lane; d < dh; d += kWave) qs[d] = q[static_cast<int64_t>(qr) * ldq + hoff + d];
  __syncthreads();
  float m = -INFINITY, l = 0.0f, o0 = 0.0f, o1 = 0.0f;
  for (int key0 = 0; key0 < L; key0 += kWave) {
    const int key = key0 + lane;
    float s = -INFINITY;
    if (key < L) {
      const float* kr = k + static_cast<int64_t>(key) * ldkv + hoff;
      float dot = 0.0f;
      for (int d = 0; d < dh; ++d) dot += qs[d] * kr[d];
      s = dot * scale;
    }
    const float m_new = fmaxf(m, wave_max(s));
    const float alpha = expf(m - m_new);
    const float pv = key < L ? expf(s - m_new) : 0.0f;
    l = l * alpha + wave_sum(pv);
    ps[lane] = pv;
    __syncthreads();
    const int nk = (L - key0) < kWave ? (L - key0) : kWave;
    float a0 = 0.0f, a1 = 0.0f;
    for (int j = 0; j < nk; ++j) {
      const float* vr = v + static_cast<int64_t>(key0 + j) * ldkv + hoff;
      if (lane < dh) a0 += ps[j] * vr[lane];
      if (lane + kWave < dh) a1 += ps[j] * vr[lane + kWave];
    }
    o0 = o0 * alpha + a0;
    o1 = o1 * alpha + a1;
    m = m_new;
    __syncthreads();
  }
  float* orow = out + static_cast<int64_t>(qr) * ldo + hoff;
  if (lane < dh) orow[lane] = o0 / l;
  if (lane + kWave < dh) orow[lane + kWave] = o1 / l;
}

hipError_t launch_gemm_f32(const char* name, int epi, const GemmF32Args& a, hipStream_t stream) {
  if (a.M <= 0) return hipSuccess;
  const dim3 grid((a.N + F32_TILE - 1) / F32_TILE, (a.M + F32_TILE - 1) / F32_TILE);
  const dim3 block(F32_TILE * F32_TILE);
  switch (epi) {
    case 0: return ECHO_LAUNCH(name, gemm_f32_nt<0>, grid, block, 0, stream, a);
    case 1: return ECHO_LAUNCH(name, gemm_f32_nt<1>, grid, block, 0, stream, a);
    default: return ECHO_LAUNCH(name, gemm_f32_nt<2>, grid, block, 0, stream, a);
  }
}

hipError_t launch_attn_f32(const float* q, int64_t ldq, const float* k, const float* v, int64_t ldkv,
                           int Mq, int L, int H, int dh, float* out, int64_t ldo, hipStream_t stream) {
  if (Mq <= 0) return hipSuccess;
  const float scale = static_cast<float>(1.0 / sqrt(static_cast<double>(dh)));
  return ECHO_LAUNCH("attn_fwd_f32", attn_fwd_f32, dim3(Mq, H), dim3(kWave), 0, stream, q, ldq, k, v,
                     ldkv, Mq, L, dh, scale, out, ldo);
}

}  // namespace echo

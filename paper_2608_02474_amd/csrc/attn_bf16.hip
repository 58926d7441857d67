// Restricted-query attention (Sec. 3.3, "Fine-grained latent-level caching"):
// the queries of the selected tokens attend over the keys and values of ALL
// tokens, per head, o = softmax(q k^T / sqrt(dh)) v, dh = 128, bf16 operands
// with fp32 accumulation and an online (streaming) softmax.
//
// gfx950 mapping.  One 256-thread workgroup = 4 waves = 128 queries of one
// head; each wave owns 32 queries.  Keys are streamed in tiles of 64 through
// LDS (K tile [key][dh] and V tile transposed to [dh][key], both
// double-buffered, 64 KB per workgroup, two workgroups per CU).
// Per tile and wave:
//   S^T (keys x queries) = K_tile . Q^T   with v_mfma_f32_32x32x16_bf16; the
//       query fragment stays in registers for the whole key loop;
//   the softmax runs per lane: each lane owns one query (its accumulator
//       column) and half of the 64 keys, so the row max/sum need one swap
//       with lane^32 only;
//   O^T (dh x queries) += V^T_tile . P^T  where P^T is the previous MFMA's
//       output converted to bf16 in registers, with no LDS round trip.
// To make P^T usable as the second MFMA's operand directly, the K rows are fed
// to the first MFMA in a permuted order (bits 2 and 3 of the row index
// swapped), so that each lane's accumulator registers hold 8 consecutive keys
// per 16-key step -- exactly the operand layout of the PV product.
// Workgroup ids are remapped so that each XCD works through a contiguous
// range of (head, query-tile) pairs: the query tiles of one head share that
// head's K/V stream in one L2.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int ATT_Q = 128, ATT_KT = 64, ATT_DH = 128, ATT_THREADS = 256;
constexpr int ATT_OS_STRIDE = ATT_DH + 8;  // output staging row (bf16), breaks bank aliasing

// swap bits 2 and 3
__device__ __forceinline__ int perm23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }
// K tile: 256-byte rows of 16 chunks; lanes reading rows perm23(l) get distinct chunks
__device__ __forceinline__ int kswz(int key, int ch) { return ch ^ perm23(key & 15); }
// V^T tile: 128-byte rows of 8 chunks
__device__ __forceinline__ int vswz(int row, int ch) { return ch ^ ((row & 7) ^ ((row >> 3) & 1)); }

__device__ __forceinline__ uint32_t half16(const uint4& v, int j) {
  const uint32_t w = (j < 2) ? v.x : (j < 4) ? v.y : (j < 6) ? v.z : v.w;
  return (j & 1) ? (w >> 16) : (w & 0xffffu);
}

__global__ void __launch_bounds__(ATT_THREADS, 2)
attn_fwd_bf16(const bf16_t* __restrict__ q, int64_t ldq, const bf16_t* __restrict__ k,
              const bf16_t* __restrict__ v, int64_t ldkv, int Mq, int L, int H, float scale_log2,
              bf16_t* __restrict__ out, int64_t ldo) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * 2 * ATT_KT * ATT_DH];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave, l32 = lane & 31, hi = lane >> 5;

  const int ntq = (Mq + ATT_Q - 1) / ATT_Q;
  const int total = ntq * H;
  int pid = blockIdx.x;
  {
    const int qq = total / 8, r = total % 8, xcd = pid % 8, loc = pid / 8;
    pid = xcd * qq + (xcd < r ? xcd : r) + loc;
  }
  const int head = pid / ntq, qt = pid % ntq;
  const int64_t hoff = static_cast<int64_t>(head) * ATT_DH;

  // query fragments: lane holds q[row][16 s + 8 hi .. +7] for the 8 k16-steps over dh
  bf16x8 qf[8];
  {
    int qr = qt * ATT_Q + wave * 32 + l32;
    qr = qr < Mq ? qr : Mq - 1;
    const bf16_t* src = q + static_cast<int64_t>(qr) * ldq + hoff + 8 * hi;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint4 u = ldg16(src + 16 * s);
      qf[s] = __builtin_bit_cast(bf16x8, u);
    }
  }

  f32x16 o[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // staging assignment: K = 4 chunks of 16 B per thread; V = 4 keys x 8 dh per thread
  const int kv_kg = tid >> 4, kv_dc = tid & 15;
  uint4 rk[4], rv[4];
  auto load_tile = [&](int key0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int id = tid + ATT_THREADS * i;
      const int key = id >> 4, ch = id & 15;
      int kg = key0 + key;
      kg = kg < L ? kg : L - 1;
      rk[i] = ldg16(k + static_cast<int64_t>(kg) * ldkv + hoff + ch * 8);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      int kg = key0 + 4 * kv_kg + u;
      kg = kg < L ? kg : L - 1;
      rv[u] = ldg16(v + static_cast<int64_t>(kg) * ldkv + hoff + kv_dc * 8);
    }
  };
  auto store_tile = [&](int stage) {
    bf16_t* Ks = smem + stage * 2 * ATT_KT * ATT_DH;
    bf16_t* Vt = Ks + ATT_KT * ATT_DH;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int id = tid + ATT_THREADS * i;
      const int key = id >> 4, ch = id & 15;
      *reinterpret_cast<uint4*>(Ks + key * ATT_DH + kswz(key, ch) * 8) = rk[i];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = kv_dc * 8 + j;  // dh
      const uint32_t lo = half16(rv[0], j) | (half16(rv[1], j) << 16);
      const uint32_t hi2 = half16(rv[2], j) | (half16(rv[3], j) << 16);
      *reinterpret_cast<uint2*>(Vt + row * ATT_KT + vswz(row, kv_kg >> 1) * 8 + (kv_kg & 1) * 4) =
          make_uint2(lo, hi2);
    }
  };

  const int nkt = (L + ATT_KT - 1) / ATT_KT;
  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nkt) load_tile((kt + 1) * ATT_KT);
    const bf16_t* Ks = smem + cur * 2 * ATT_KT * ATT_DH;
    const bf16_t* Vt = Ks + ATT_KT * ATT_DH;

    // S^T = K . Q^T for two 32-key blocks
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.0f;
      const int key = kb * 32 + perm23(l32);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(Ks + key * ATT_DH + kswz(key, 2 * s + hi) * 8);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[kb], 0, 0, 0);
      }
    }

    // online softmax; register r of block kb holds key kb*32 + 16(r/8) + 8hi + r%8
    const int key0 = kt * ATT_KT;
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kg = key0 + kb * 32 + 16 * (r >> 3) + 8 * hi + (r & 7);
        const float sv = kg < L ? sacc[kb][r] * scale_log2 : -INFINITY;
        sacc[kb][r] = sv;
        mx = fmaxf(mx, sv);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float psum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = __builtin_amdgcn_exp2f(sacc[kb][r] - m_new);
        sacc[kb][r] = pv;
        psum += pv;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[d][r] *= alpha;

    bf16x8 pf[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int j = 0; j < 8; ++j) pf[kb][a][j] = static_cast<__bf16>(sacc[kb][8 * a + j]);

    // O^T += V^T . P^T
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int row = d * 32 + l32;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
          const int ch = 4 * kb + 2 * a + hi;
          const bf16x8 va = *reinterpret_cast<const bf16x8*>(Vt + row * ATT_KT + vswz(row, ch) * 8);
          o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pf[kb][a], o[d], 0, 0, 0);
        }
    }

    if (kt + 1 < nkt) store_tile(cur ^ 1);
    __syncthreads();
  }

  // normalise and write through LDS so that global stores are full 16-byte rows
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.0f / l_tot;
  bf16_t* Os = smem;  // [128][ATT_OS_STRIDE], free after the final barrier
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int dh = d * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
      Os[(wave * 32 + l32) * ATT_OS_STRIDE + dh] = f32_to_bf16(o[d][r] * inv);
    }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < (ATT_Q * ATT_DH / 8) / ATT_THREADS; ++i) {
    const int id = tid + ATT_THREADS * i;
    const int row = id >> 4, ch = id & 15;
    const int qr = qt * ATT_Q + row;
    if (qr < Mq)
      stg16(out + static_cast<int64_t>(qr) * ldo + hoff + ch * 8,
            *reinterpret_cast<const uint4*>(Os + row * ATT_OS_STRIDE + ch * 8));
  }
}

hipError_t launch_attn_bf16(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                            int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                            hipStream_t stream) {
  if (Mq <= 0) return hipSuccess;
  const float scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(ATT_DH)));
  const int ntq = (Mq + ATT_Q - 1) / ATT_Q;
  return ECHO_LAUNCH("attn_fwd_bf16", attn_fwd_bf16, dim3(ntq * H), dim3(ATT_THREADS), 0, stream, q,
                     ldq, k, v, ldkv, Mq, L, H, scale_log2, out, ldo);
}

}  // namespace echo

// Adaptive reference cache (Sec. 3.4, "Memory-efficient Cache Management"):
// a fresh output whose cosine similarity with its chain's current reference
// exceeds tau is stored as an int8 residual against it, otherwise it becomes
// a new full-precision reference; references nobody holds are released.
//
// Chains are the tokens of one spatial row of the latent grid (chain_len
// consecutive indices) and keep their current reference across writes.
// References live in a pool of `capacity` rows with a hold count per slot and
// a stack of free slots.  One update is four launches on one stream:
//   refcache_release  one thread per rewritten token: drop the hold of its old
//                     entry; a slot whose count reaches zero goes back on the
//                     free stack (pushes only);
//   refcache_write    one workgroup per chain: scan the chain's rewritten
//                     tokens in index order, keeping the current reference
//                     row in registers; fp64 similarity, int8 residual or new
//                     reference (pops only; a chain's old reference that only
//                     the chain still held is reused in place);
//   refcache_fuse     one wave per row: fresh rows output cast(y_sel) and
//                     record their input as the saliency reference; the
//                     others are rebuilt from their entry (16-byte accesses).
// Every live slot is held by a token entry or a chain, so capacity >= L +
// number of chains never runs out.  Slot numbers depend on the order of the
// atomic pops; stored values and decisions do not.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kRcThreads = 256;
constexpr int kRcWaves = kRcThreads / kWave;

__global__ void __launch_bounds__(256)
refcache_init(int L, int n_chains, int capacity, int32_t* __restrict__ refcount,
              int32_t* __restrict__ free_list, int32_t* __restrict__ free_top,
              int32_t* __restrict__ chain_ref, int32_t* __restrict__ ent_slot,
              uint8_t* __restrict__ ent_kind, float* __restrict__ scale) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < capacity) {
    refcount[i] = 0;
    free_list[i] = static_cast<int32_t>(i);
  }
  if (i < L) {
    ent_slot[i] = -1;
    ent_kind[i] = 0;
    scale[i] = 0.0f;
  }
  if (i < n_chains) chain_ref[i] = -1;
  if (i == 0) *free_top = capacity;
}

__global__ void __launch_bounds__(256)
refcache_release(const int32_t* __restrict__ idx, int n_sel, int32_t* __restrict__ refcount,
                 int32_t* __restrict__ free_list, int32_t* __restrict__ free_top,
                 int32_t* __restrict__ ent_slot, uint8_t* __restrict__ ent_kind) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n_sel) return;
  const int l = idx[j];
  if (ent_kind[l] == 0) return;
  const int s = ent_slot[l];
  if (atomicSub(&refcount[s], 1) == 1) free_list[atomicAdd(free_top, 1)] = s;
  ent_kind[l] = 0;
  ent_slot[l] = -1;
}

// sum over the workgroup; every thread gets the result
template <typename T>
__device__ __forceinline__ T block_sum(T v, T* red) {
  v = wave_sum(v);
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  T s = red[0];
#pragma unroll
  for (int w = 1; w < kRcWaves; ++w) s += red[w];
  return s;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int w = 1; w < kRcWaves; ++w) s = fmaxf(s, red[w]);
  return s;
}

// fp32(a - b) and fp32(fp32(a * b) + c) as separate IEEE operations
__device__ __forceinline__ float sub_rn(float a, float b) {
#pragma clang fp contract(off)
  return a - b;
}
__device__ __forceinline__ float mul_add_rn(float a, float b, float c) {
#pragma clang fp contract(off)
  return a * b + c;
}

template <typename T> __device__ __forceinline__ float rc_round(float v);
template <> __device__ __forceinline__ float rc_round<float>(float v) { return v; }
template <> __device__ __forceinline__ float rc_round<bf16_t>(float v) { return bf16_to_f32(f32_to_bf16(v)); }

// One workgroup per chain.  Thread t owns elements 4 t + 1024 u (u < U) of
// a row; D <= 1024 U, D % 4 == 0.
template <typename T, int U>
__global__ void __launch_bounds__(kRcThreads)
refcache_write(const int32_t* __restrict__ idx, int n_sel, const float* __restrict__ y_sel, int D,
               int chain_len, float tau, T* __restrict__ pool, int32_t* __restrict__ refcount,
               const int32_t* __restrict__ free_list, int32_t* __restrict__ free_top,
               int32_t* __restrict__ chain_ref, int32_t* __restrict__ ent_slot,
               uint8_t* __restrict__ ent_kind, int8_t* __restrict__ codes, float* __restrict__ scale) {
  __shared__ double red_d[2][kRcWaves];
  __shared__ float red_f[kRcWaves];
  __shared__ int sh_slot;
  const int c = blockIdx.x;
  const int tid = threadIdx.x;
  const int lo = c * chain_len, hi = lo + chain_len;
  // rewritten tokens of this chain: idx[j0 .. j1) (idx ascending)
  int a = 0, b = n_sel;
  while (a < b) { const int m = (a + b) >> 1; if (idx[m] < lo) a = m + 1; else b = m; }
  const int j0 = a;
  b = n_sel;
  while (a < b) { const int m = (a + b) >> 1; if (idx[m] < hi) a = m + 1; else b = m; }
  const int j1 = a;
  if (j0 == j1) return;

  int cr = chain_ref[c];
  float r[U][4];                      // current reference row (stored values)
  double rr = 0.0;                    // its squared norm
  auto col = [&](int u) { return 4 * tid + 1024 * u; };
  if (cr >= 0) {
    const T* rp = pool + static_cast<int64_t>(cr) * D;
    double s = 0.0;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        r[u][e] = col(u) < D ? Elem<T>::load(rp, col(u) + e) : 0.0f;
        s += static_cast<double>(r[u][e]) * r[u][e];
      }
    rr = block_sum(s, red_d[0]);
  }

  float y[U][4];
  float4 ynext[U];  // the next token's row, loaded while this one is processed
  auto fetch = [&](int j) __attribute__((always_inline)) {
    const float* yp = y_sel + static_cast<int64_t>(j) * D;
#pragma unroll
    for (int u = 0; u < U; ++u)
      ynext[u] = col(u) < D ? *reinterpret_cast<const float4*>(yp + col(u)) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  };
  fetch(j0);
  for (int j = j0; j < j1; ++j) {
    const int l = idx[j];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      y[u][0] = ynext[u].x; y[u][1] = ynext[u].y; y[u][2] = ynext[u].z; y[u][3] = ynext[u].w;
    }
    if (j + 1 < j1) fetch(j + 1);
    bool residual = false;
    if (cr >= 0) {
      double dot = 0.0, yy = 0.0;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dot += static_cast<double>(y[u][e]) * r[u][e];
          yy += static_cast<double>(y[u][e]) * y[u][e];
        }
      dot = block_sum(dot, red_d[0]);
      yy = block_sum(yy, red_d[1]);
      const double sim = (yy == 0.0 || rr == 0.0) ? 0.0 : dot / (sqrt(yy) * sqrt(rr));
      residual = sim > static_cast<double>(tau);
    }
    if (residual) {
      float res[U][4];
      float amax = 0.0f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          res[u][e] = sub_rn(y[u][e], r[u][e]);
          amax = fmaxf(amax, fabsf(res[u][e]));
        }
      amax = block_max(amax, red_f);
      const bool nz = amax > 0.0f;
      const float inv = nz ? __fdiv_rn(127.0f, amax) : 0.0f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (col(u) >= D) continue;
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float q = rintf(__fmul_rn(res[u][e], inv));
          q = fminf(fmaxf(q, -127.0f), 127.0f);
          word |= (static_cast<uint32_t>(static_cast<int32_t>(q)) & 0xffu) << (8 * e);
        }
        *reinterpret_cast<uint32_t*>(codes + static_cast<int64_t>(l) * D + col(u)) = word;
      }
      if (tid == 0) {
        scale[l] = nz ? __fdiv_rn(amax, 127.0f) : 0.0f;
        ent_kind[l] = 2;
        ent_slot[l] = cr;
        refcount[cr] += 1;  // only this chain's tokens hold its references
      }
    } else {
      // new reference: the chain's old one is reused in place when only the
      // chain held it, otherwise the chain lets go of it and a slot is popped
      if (tid == 0) {
        int s;
        if (cr >= 0 && refcount[cr] == 1) {
          s = cr;
        } else {
          const int top = atomicSub(free_top, 1);
          if (top > 0) {
            s = free_list[top - 1];
            if (cr >= 0) refcount[cr] -= 1;
          } else {
            // cannot happen with capacity >= L + chains; kept so that a broken
            // invariant leaves the token without an entry instead of writing
            // outside the pool
            atomicAdd(free_top, 1);
            s = -1;
          }
        }
        if (s >= 0) {
          refcount[s] = 2;  // the token's entry and the chain
          ent_kind[l] = 1;
          ent_slot[l] = s;
          scale[l] = 0.0f;
          chain_ref[c] = s;
        }
        sh_slot = s;
      }
      __syncthreads();
      if (sh_slot < 0) continue;
      cr = sh_slot;
      T* rp = pool + static_cast<int64_t>(cr) * D;
      double s = 0.0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          r[u][e] = rc_round<T>(y[u][e]);
          s += static_cast<double>(r[u][e]) * r[u][e];
          if (col(u) < D) Elem<T>::store(rp, col(u) + e, r[u][e]);
        }
      }
      rr = block_sum(s, red_d[0]);
    }
  }
}

// waves [0, n_sel): fresh row idx[j]; waves [n_sel, n_sel + L): row i reads
// its entry if mask[i] == 0.  8-element chunks with 16-byte accesses, four
// chunks' loads issued before any is used.
template <typename T>
__global__ void __launch_bounds__(kRcThreads)
refcache_fuse(const T* __restrict__ x, const int32_t* __restrict__ idx, const uint8_t* __restrict__ mask,
              int n_sel, int L, int D, const float* __restrict__ y_sel, const T* __restrict__ pool,
              const int32_t* __restrict__ ent_slot, const uint8_t* __restrict__ ent_kind,
              const int8_t* __restrict__ codes, const float* __restrict__ scale, T* __restrict__ xref,
              T* __restrict__ y) {
  constexpr int B = 4;  // chunks in flight per lane
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kRcWaves + wave;
  const int nch = D / 8;
  if (g < n_sel) {
    const int64_t i = idx[g];
    const float* ys = y_sel + g * D;
    for (int c0 = lane; c0 < nch; c0 += B * kWave) {
      Raw8<float> yr[B];
      Raw8<T> xr[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int c = c0 + u * kWave;
        if (c < nch) {
          yr[u].load(ys + c * 8);
          xr[u].load(x + i * D + c * 8);
        }
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int c = c0 + u * kWave;
        if (c < nch) {
          float v[8];
          yr[u].unpack(v);
          stg16(y + i * D + c * 8, pack16(v, static_cast<const T*>(nullptr)));
          if (sizeof(T) == 4) stg16(y + i * D + c * 8 + 4, pack16(v + 4, static_cast<const T*>(nullptr)));
          xr[u].store(xref + i * D + c * 8);
        }
      }
    }
    return;
  }
  const int64_t i = g - n_sel;
  if (i >= L || mask[i]) return;
  const int kind = ent_kind[i];
  const T* rp = pool + static_cast<int64_t>(ent_slot[i] < 0 ? 0 : ent_slot[i]) * D;
  const float sc = scale[i];
  for (int c0 = lane; c0 < nch; c0 += B * kWave) {
    Raw8<T> rr[B];
    uint2 cw[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int c = c0 + u * kWave;
      if (c < nch && kind != 0) {
        rr[u].load(rp + c * 8);
        cw[u] = *reinterpret_cast<const uint2*>(codes + i * D + c * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int c = c0 + u * kWave;
      if (c >= nch) continue;
      float v[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
      if (kind != 0) rr[u].unpack(v);
      if (kind == 2) {
        const uint32_t w[2] = {cw[u].x, cw[u].y};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int8_t q = static_cast<int8_t>((w[e / 4] >> (8 * (e % 4))) & 0xffu);
          v[e] = mul_add_rn(sc, static_cast<float>(q), v[e]);
        }
      }
      stg16(y + i * D + c * 8, pack16(v, static_cast<const T*>(nullptr)));
      if (sizeof(T) == 4) stg16(y + i * D + c * 8 + 4, pack16(v + 4, static_cast<const T*>(nullptr)));
    }
  }
}

hipError_t launch_refcache_init(int L, int n_chains, int capacity, int32_t* refcount, int32_t* free_list,
                                int32_t* free_top, int32_t* chain_ref, int32_t* ent_slot, uint8_t* ent_kind,
                                float* scale, hipStream_t stream) {
  const int n = capacity > L ? capacity : L;
  return ECHO_LAUNCH("refcache_init", refcache_init, dim3((n + 255) / 256), dim3(256), 0, stream, L,
                     n_chains, capacity, refcount, free_list, free_top, chain_ref, ent_slot, ent_kind, scale);
}

template <typename T>
static hipError_t refcache_update_t(const T* x, const int32_t* idx, const uint8_t* mask, int n_sel, int L, int D,
                                    int chain_len, float tau, const float* y_sel, T* pool, int32_t* refcount,
                                    int32_t* free_list, int32_t* free_top, int32_t* chain_ref, int32_t* ent_slot,
                                    uint8_t* ent_kind, int8_t* codes, float* scale, T* xref, T* y,
                                    hipStream_t stream) {
  const int n_chains = L / chain_len;
  TimedLaunch scope("refcache_update", stream);
  if (n_sel > 0) {
    hipLaunchKernelGGL(refcache_release, dim3((n_sel + 255) / 256), dim3(256), 0, stream, idx, n_sel, refcount,
                       free_list, free_top, ent_slot, ent_kind);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int U = (D + 1023) / 1024;
#define ECHO_RC_CASE(UU)                                                                                   \
    if (U <= UU) {                                                                                         \
      hipLaunchKernelGGL((refcache_write<T, UU>), dim3(n_chains), dim3(kRcThreads), 0, stream, idx, n_sel,  \
                         y_sel, D, chain_len, tau, pool, refcount, free_list, free_top, chain_ref, ent_slot, \
                         ent_kind, codes, scale);                                                          \
    } else
    ECHO_RC_CASE(1) ECHO_RC_CASE(2) ECHO_RC_CASE(4) ECHO_RC_CASE(5) ECHO_RC_CASE(8) ECHO_RC_CASE(16) {
      return hipErrorInvalidValue;
    }
#undef ECHO_RC_CASE
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t waves = static_cast<int64_t>(n_sel) + L;
  hipLaunchKernelGGL((refcache_fuse<T>), dim3(static_cast<unsigned>((waves + kRcWaves - 1) / kRcWaves)),
                     dim3(kRcThreads), 0, stream, x, idx, mask, n_sel, L, D, y_sel, pool, ent_slot, ent_kind,
                     codes, scale, xref, y);
  return hipGetLastError();
}

hipError_t launch_refcache_update(int dtype_bf16, const void* x, const int32_t* idx, const uint8_t* mask,
                                  int n_sel, int L, int D, int chain_len, float tau, const float* y_sel,
                                  void* pool, int32_t* refcount, int32_t* free_list, int32_t* free_top,
                                  int32_t* chain_ref, int32_t* ent_slot, uint8_t* ent_kind, int8_t* codes,
                                  float* scale, void* xref, void* y, hipStream_t stream) {
  if (dtype_bf16)
    return refcache_update_t<bf16_t>(static_cast<const bf16_t*>(x), idx, mask, n_sel, L, D, chain_len, tau,
                                     y_sel, static_cast<bf16_t*>(pool), refcount, free_list, free_top, chain_ref,
                                     ent_slot, ent_kind, codes, scale, static_cast<bf16_t*>(xref),
                                     static_cast<bf16_t*>(y), stream);
  return refcache_update_t<float>(static_cast<const float*>(x), idx, mask, n_sel, L, D, chain_len, tau, y_sel,
                                  static_cast<float*>(pool), refcount, free_list, free_top, chain_ref, ent_slot,
                                  ent_kind, codes, scale, static_cast<float*>(xref), static_cast<float*>(y),
                                  stream);
}

}  // namespace echo

// Modulated LayerNorm of token rows (the adaLN "LN(z) * (1 + scale) + shift"
// in front of attention and FFN of the DiT block, Sec. 3.3).
//
// One wave per row; the row is held in registers (8-element chunks, all
// non-temporal loads issued before the first is used; the output keeps
// ordinary stores, since the GEMM after it reads it), mean and biased
// variance are reduced in
// fp32 with two passes over the registers, and the modulated result is
// written in the output storage type.  Every access, the modulation vectors
// included, is a 16-byte vector load or store.  Rows longer than 512 * MAXC
// elements take the MAXC == 0 variant, which re-reads the row.  fp32 rows
// (the second LayerNorm) of width 2048, 4096 or 5120 are shared by the waves
// of a workgroup instead (modln_rows_wg).
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kLnThreads = 256;
constexpr int kLnWaves = kLnThreads / kWave;

__device__ __forceinline__ void ln_load8(const float* p, float* v) {
  unpack16(ldg16(p), v, static_cast<const float*>(nullptr));
  unpack16(ldg16(p + 4), v + 4, static_cast<const float*>(nullptr));
}
__device__ __forceinline__ void ln_load8(const bf16_t* p, float* v) {
  unpack16(ldg16(p), v, static_cast<const bf16_t*>(nullptr));
}
__device__ __forceinline__ void ln_store8(float* p, const float* v) {
  stg16(p, pack16(v, static_cast<const float*>(nullptr)));
  stg16(p + 4, pack16(v + 4, static_cast<const float*>(nullptr)));
}
__device__ __forceinline__ void ln_store8(bf16_t* p, const float* v) {
  stg16(p, pack16(v, static_cast<const bf16_t*>(nullptr)));
}

template <typename Tin, typename Tout, int MAXC>
__global__ void __launch_bounds__(kLnThreads)
modln_rows(const Tin* __restrict__ x, int M, int D, const float* __restrict__ shift,
           const float* __restrict__ scale, float eps, Tout* __restrict__ out) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kLnWaves + wave;
  if (row >= M) return;
  const Tin* xr = x + row * D;
  Tout* orow = out + row * D;
  const int nch = D / 8;
  const float invD = 1.0f / static_cast<float>(D);
  if (MAXC > 0) {
    // every load of the row is issued before any of them is used; lanes past
    // the row end re-load its last chunk (in bounds) and add nothing
    constexpr int R = MAXC > 0 ? MAXC : 1;
    auto body = [&](auto full_c) __attribute__((always_inline)) {
      constexpr bool FULL = decltype(full_c)::value;  // every lane owns R chunks
      Raw8<Tin> raw[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        raw[u].load_nt(xr + (FULL || c < nch ? c : nch - 1) * 8);
      }
      float sum = 0.0f;
#pragma unroll
      for (int u = 0; u < R; ++u) {
        float v[8];
        raw[u].unpack(v);
        const bool ok = FULL || lane + u * kWave < nch;
#pragma unroll
        for (int j = 0; j < 8; ++j) sum += ok ? v[j] : 0.0f;
      }
      const float mean = wave_sum(sum) * invD;
      float sq = 0.0f;
#pragma unroll
      for (int u = 0; u < R; ++u) {
        float v[8];
        raw[u].unpack(v);
        const bool ok = FULL || lane + u * kWave < nch;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float d = v[j] - mean;
          sq += ok ? d * d : 0.0f;
        }
      }
      const float rstd = 1.0f / sqrtf(wave_sum(sq) * invD + eps);
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        if (FULL || c < nch) {
          float v[8], o[8], sc[8], sh[8];
          raw[u].unpack(v);
          ln_load8(scale + c * 8, sc);
          ln_load8(shift + c * 8, sh);
#pragma unroll
          for (int j = 0; j < 8; ++j) o[j] = (v[j] - mean) * rstd * (1.0f + sc[j]) + sh[j];
          ln_store8(orow + c * 8, o);
        }
      }
    };
    if (nch == R * kWave)
      body(std::integral_constant<bool, true>{});
    else
      body(std::integral_constant<bool, false>{});
  } else {
    float sum = 0.0f;
    for (int c = lane; c < nch; c += kWave) {
      float v[8];
      ln_load8(xr + c * 8, v);
#pragma unroll
      for (int j = 0; j < 8; ++j) sum += v[j];
    }
    const float mean = wave_sum(sum) * invD;
    float sq = 0.0f;
    for (int c = lane; c < nch; c += kWave) {
      float v[8];
      ln_load8(xr + c * 8, v);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[j] - mean;
        sq += d * d;
      }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(sq) * invD + eps);
    for (int c = lane; c < nch; c += kWave) {
      float v[8], o[8], sc[8], sh[8];
      ln_load8(xr + c * 8, v);
      ln_load8(scale + c * 8, sc);
      ln_load8(shift + c * 8, sh);
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (v[j] - mean) * rstd * (1.0f + sc[j]) + sh[j];
      ln_store8(orow + c * 8, o);
    }
  }
}

// An empty asm that claims to change the raw row registers, so that later
// unpacks are recomputed rather than kept live from earlier passes.
template <int R>
__device__ __forceinline__ void raw_fence(Raw8<bf16_t> (&raw)[R]) {
#pragma unroll
  for (int u = 0; u < R; ++u) asm volatile("" : "+v"(raw[u].v.x), "+v"(raw[u].v.y), "+v"(raw[u].v.z), "+v"(raw[u].v.w));
}
template <int R>
__device__ __forceinline__ void raw_fence(Raw8<float> (&raw)[R]) {
#pragma unroll
  for (int u = 0; u < R; ++u) {
    asm volatile("" : "+v"(raw[u].v0.x), "+v"(raw[u].v0.y), "+v"(raw[u].v0.z), "+v"(raw[u].v0.w));
    asm volatile("" : "+v"(raw[u].v1.x), "+v"(raw[u].v1.y), "+v"(raw[u].v1.z), "+v"(raw[u].v1.w));
  }
}

// The same LayerNorm with the modulation vectors staged once per workgroup in
// LDS (1 + scale, then shift: 8 D bytes) and each wave looping over rows
// (row = 4 * blockIdx.x + wave, then in steps of 4 * gridDim.x).  Reading the
// two vectors from L2 for every row used to move four times the row's own
// bytes through the load path; from LDS they cost two 16-byte reads per
// eight elements.  Requires MAXC > 0 and D <= kLnLdsMaxD.
constexpr int kLnLdsMaxD = 8192;

template <typename Tin, typename Tout, int MAXC, bool FULL_ROWS>
__global__ void __launch_bounds__(kLnThreads)
modln_rows_lds(const Tin* __restrict__ x, int M, int D, const float* __restrict__ shift,
               const float* __restrict__ scale, float eps, Tout* __restrict__ out) {
  extern __shared__ float4 lds_mod4[];
  float* s1 = reinterpret_cast<float*>(lds_mod4);  // [D] 1 + scale
  float* sh = s1 + D;                              // [D] shift
  for (int i = threadIdx.x; i < D / 4; i += kLnThreads) {
    float4 a = reinterpret_cast<const float4*>(scale)[i];
    a.x += 1.0f;
    a.y += 1.0f;
    a.z += 1.0f;
    a.w += 1.0f;
    reinterpret_cast<float4*>(s1)[i] = a;
    reinterpret_cast<float4*>(sh)[i] = reinterpret_cast<const float4*>(shift)[i];
  }
  __syncthreads();
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nch = D / 8;
  const float invD = 1.0f / static_cast<float>(D);
  constexpr int R = MAXC;
  auto body = [&](auto full_c, const Tin* xr, Tout* orow) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_c)::value;  // every lane owns R chunks
    Raw8<Tin> raw[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int c = lane + u * kWave;
      raw[u].load_nt(xr + (FULL || c < nch ? c : nch - 1) * 8);
    }
    float sum = 0.0f;
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float v[8];
      raw[u].unpack(v);
      const bool ok = FULL || lane + u * kWave < nch;
#pragma unroll
      for (int j = 0; j < 8; ++j) sum += ok ? v[j] : 0.0f;
    }
    const float mean = wave_sum(sum) * invD;
    float sq = 0.0f;
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float v[8];
      raw[u].unpack(v);
      const bool ok = FULL || lane + u * kWave < nch;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[j] - mean;
        sq += ok ? d * d : 0.0f;
      }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(sq) * invD + eps);
    // unpack again below rather than keep the first passes' floats live, and
    // take one chunk at a time (hoisting every chunk's modulation reads ahead
    // of the first store doubles the registers)
    raw_fence(raw);
#pragma unroll
    for (int u = 0; u < R; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      const int c = lane + u * kWave;
      if (FULL || c < nch) {
        float v[8], o[8], sc[8], shv[8];
        raw[u].unpack(v);
        const float4* a = reinterpret_cast<const float4*>(s1 + c * 8);
        const float4* b = reinterpret_cast<const float4*>(sh + c * 8);
        const float4 a0 = a[0], a1 = a[1], b0 = b[0], b1 = b[1];
        sc[0] = a0.x; sc[1] = a0.y; sc[2] = a0.z; sc[3] = a0.w;
        sc[4] = a1.x; sc[5] = a1.y; sc[6] = a1.z; sc[7] = a1.w;
        shv[0] = b0.x; shv[1] = b0.y; shv[2] = b0.z; shv[3] = b0.w;
        shv[4] = b1.x; shv[5] = b1.y; shv[6] = b1.z; shv[7] = b1.w;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = (v[j] - mean) * rstd * sc[j] + shv[j];
        ln_store8(orow + c * 8, o);
      }
    }
  };
  // FULL_ROWS (D = 512 MAXC): every lane owns MAXC chunks.  A kernel of its
  // own, so that the registers of the ragged case do not count against it
  // (LN1 186 -> 140, LN2 172 -> 124 registers at D = 5120).
  const int64_t step = static_cast<int64_t>(gridDim.x) * kLnWaves;
  for (int64_t row = static_cast<int64_t>(blockIdx.x) * kLnWaves + wave; row < M; row += step)
    body(std::integral_constant<bool, FULL_ROWS>{}, x + row * D, out + row * D);
}


// fp32 rows (the second LayerNorm, over x1) are shared by a workgroup instead:
// WAVES = D / 512 waves, each thread one 8-element chunk (c = threadIdx.x),
// whose modulation it keeps in registers for every row it takes.  The
// workgroup loops over rows and issues the next row's loads before the
// current row's two reductions (each a wave sum, then the WAVES partial sums
// added in wave order from LDS).  With a wave per row (the kernel above) each
// wave keeps 20 KB of a 5120-wide fp32 row in flight and the second LayerNorm
// ran at 0.67 of HBM; this form keeps 32 bytes per thread and the next row
// in flight (75.3 -> 71.1 us on 13104 x 5120 rows, 0.71 of HBM).  It does not
// help bf16 rows (the first LayerNorm).
template <typename Tin, typename Tout, int WAVES>
__global__ void __launch_bounds__(WAVES * 64)
modln_rows_wg(const Tin* __restrict__ x, int M, int D, const float* __restrict__ shift,
              const float* __restrict__ scale, float eps, Tout* __restrict__ out) {
  __shared__ float red[2][WAVES];  // per-wave partial sums: [0] the row sum, [1] the squared deviations
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const float invD = 1.0f / static_cast<float>(D);
  float a[8], b[8];
  ln_load8(scale + tid * 8, a);
  ln_load8(shift + tid * 8, b);
#pragma unroll
  for (int j = 0; j < 8; ++j) a[j] += 1.0f;
  int row = blockIdx.x;  // gridDim.x <= M
  Raw8<Tin> cur, nxt;
  cur.load_nt(x + static_cast<int64_t>(row) * D + tid * 8);
  for (; row < M; row += gridDim.x) {
    const int nrow = row + gridDim.x;
    if (nrow < M) nxt.load_nt(x + static_cast<int64_t>(nrow) * D + tid * 8);
    float v[8];
    cur.unpack(v);
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += v[j];
    s = wave_sum(s);
    if (lane == 0) red[0][wave] = s;
    // (a slot is written again only after the next barrier, which every
    // reader of this row's value reaches after its read)
    __syncthreads();
    s = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) s += red[0][w];
    const float mean = s * invD;
    float sq = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float d = v[j] - mean;
      sq += d * d;
    }
    sq = wave_sum(sq);
    if (lane == 0) red[1][wave] = sq;
    __syncthreads();
    sq = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) sq += red[1][w];
    const float rstd = 1.0f / sqrtf(sq * invD + eps);
    float o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = (v[j] - mean) * rstd * a[j] + b[j];
    ln_store8(out + static_cast<int64_t>(row) * D + tid * 8, o);
    cur = nxt;
  }
}

template <typename Tin, typename Tout, int WAVES>
static hipError_t launch_modln_wg(const char* name, const Tin* x, int M, int D, const float* shift,
                                  const float* scale, float eps, Tout* out, hipStream_t stream) {
  // about 20 waves per CU (two workgroups at D = 5120: one or three were slower)
  const int per_cu = 20 / WAVES;
  const int cap = per_cu * device_cu_count();
  const dim3 grid(static_cast<unsigned>(M < cap ? M : cap));
  return ECHO_LAUNCH(name, (modln_rows_wg<Tin, Tout, WAVES>), grid, dim3(WAVES * 64), 0, stream, x, M, D,
                     shift, scale, eps, out);
}

template <typename Tin, typename Tout>
static hipError_t launch_modln_t(const char* name, const Tin* x, int M, int D, const float* shift,
                                 const float* scale, float eps, Tout* out, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (std::is_same<Tin, float>::value) {
    // the widths built (and tested): 2048, 4096 and 5120
    if (D == 512 * 4) return launch_modln_wg<Tin, Tout, 4>(name, x, M, D, shift, scale, eps, out, stream);
    if (D == 512 * 8) return launch_modln_wg<Tin, Tout, 8>(name, x, M, D, shift, scale, eps, out, stream);
    if (D == 512 * 10) return launch_modln_wg<Tin, Tout, 10>(name, x, M, D, shift, scale, eps, out, stream);
  }
  const dim3 grid((M + kLnWaves - 1) / kLnWaves);
  const int per_lane = (D / 8 + kWave - 1) / kWave;
  if (D <= kLnLdsMaxD) {
    // four workgroups per CU (the LDS of the modulation vectors allows four
    // at the largest D), each wave looping over its rows
    const int cap = 4 * device_cu_count();
    const dim3 grid_l(static_cast<unsigned>(grid.x < static_cast<unsigned>(cap) ? grid.x : cap));
    const size_t lds = sizeof(float) * 2 * static_cast<size_t>(D);
#define ECHO_LNL_CASE(MC)                                                                              \
  if (per_lane <= MC) {                                                                                \
    if (D == 512 * MC)                                                                                 \
      return ECHO_LAUNCH(name, (modln_rows_lds<Tin, Tout, MC, true>), grid_l, dim3(kLnThreads), lds, stream, x, \
                         M, D, shift, scale, eps, out);                                                \
    return ECHO_LAUNCH(name, (modln_rows_lds<Tin, Tout, MC, false>), grid_l, dim3(kLnThreads), lds, stream, x,  \
                       M, D, shift, scale, eps, out);                                                  \
  }
    ECHO_LNL_CASE(1)
    ECHO_LNL_CASE(2)
    ECHO_LNL_CASE(3)
    ECHO_LNL_CASE(4)
    ECHO_LNL_CASE(6)
    ECHO_LNL_CASE(8)
    ECHO_LNL_CASE(10)
    ECHO_LNL_CASE(12)
    ECHO_LNL_CASE(16)
#undef ECHO_LNL_CASE
  }
#define ECHO_LN_CASE(MC)                                                                       \
  if (per_lane <= MC)                                                                          \
    return ECHO_LAUNCH(name, (modln_rows<Tin, Tout, MC>), grid, dim3(kLnThreads), 0, stream, x, \
                       M, D, shift, scale, eps, out);
  ECHO_LN_CASE(1)
  ECHO_LN_CASE(2)
  ECHO_LN_CASE(3)
  ECHO_LN_CASE(4)
  ECHO_LN_CASE(6)
  ECHO_LN_CASE(8)
  ECHO_LN_CASE(10)
  ECHO_LN_CASE(12)
  ECHO_LN_CASE(16)
#undef ECHO_LN_CASE
  return ECHO_LAUNCH(name, (modln_rows<Tin, Tout, 0>), grid, dim3(kLnThreads), 0, stream, x, M, D,
                     shift, scale, eps, out);
}

// LN1 over the block input rows (bf16 -> bf16, or f32 -> f32).
hipError_t launch_modln_input(int dtype_bf16, const void* x, int M, int D, const float* shift,
                              const float* scale, float eps, void* out, hipStream_t stream) {
  if (dtype_bf16)
    return launch_modln_t<bf16_t, bf16_t>("modln_in_bf16", static_cast<const bf16_t*>(x), M, D, shift,
                                          scale, eps, static_cast<bf16_t*>(out), stream);
  return launch_modln_t<float, float>("modln_in_f32", static_cast<const float*>(x), M, D, shift, scale,
                                      eps, static_cast<float*>(out), stream);
}

// LN2 over the fp32 attention-residual rows x1 (-> bf16 or f32).
hipError_t launch_modln_x1(int dtype_bf16, const float* x1, int M, int D, const float* shift,
                           const float* scale, float eps, void* out, hipStream_t stream) {
  if (dtype_bf16)
    return launch_modln_t<float, bf16_t>("modln_x1_bf16", x1, M, D, shift, scale, eps,
                                         static_cast<bf16_t*>(out), stream);
  return launch_modln_t<float, float>("modln_x1_f32", x1, M, D, shift, scale, eps,
                                      static_cast<float*>(out), stream);
}

}  // namespace echo

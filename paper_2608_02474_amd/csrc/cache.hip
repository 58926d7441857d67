// Int8 residual cache write and mask fusion (Sec. 3.3: output = m * fresh +
// (1 - m) * cached; Sec. 3.4: cached = reference + dequantized int8 residual,
// cast back to the compute precision).
//
// One launch, one wave per row:
//   waves [0, n_sel)        recomputed row i = idx[j]: res = y_sel[j] - x_i in
//                           fp32, absmax, per-row scale, int8 codes, reference
//                           := x_i, output := cast(y_sel[j]);
//   waves [n_sel, n_sel+L)  row i = wave - n_sel, if mask[i] == 0: output :=
//                           cast(xref_i + scale_i * code).
// Rows are streamed with 16-byte non-temporal loads/stores (8 elements per
// chunk; nothing written here is read again before the next step), every
// load of a row issued before the first is used; the fresh row's y and x stay
// in registers between the absmax and the quantization.
// Every fp32 step is a separately rounded IEEE operation (no fused
// multiply-add), so codes and reused rows are exactly the fp32 values the
// definition gives.
//
// Codecs of the module ablation (Table 2), one template parameter:
//   kResidualInt8  the cache above (reference x_i, int8 residual y - x_i);
//   kFull          the output itself in the activation dtype: a fresh row
//                  also goes to `store`, a reused row is copied from it;
//   kNaiveInt8     int8 codes of y itself (no reference), read back as
//                  cast(fp32(scale * code)).
// Every codec records xref_i := x_i for a fresh row (the saliency reference).
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kCacheThreads = 256;
constexpr int kCacheWavesPerBlock = kCacheThreads / kWave;
constexpr int kResidualInt8 = 0, kFull = 1, kNaiveInt8 = 2;

__device__ __forceinline__ void load8(const float* p, float* v) {
  const uint4 a = ldg16(p), b = ldg16(p + 4);
  unpack16(a, v, static_cast<const float*>(nullptr));
  unpack16(b, v + 4, static_cast<const float*>(nullptr));
}
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
  unpack16(ldg16(p), v, static_cast<const bf16_t*>(nullptr));
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  stg16_nt(p, pack16(v, static_cast<const float*>(nullptr)));
  stg16_nt(p + 4, pack16(v + 4, static_cast<const float*>(nullptr)));
}
__device__ __forceinline__ void store8(bf16_t* p, const float* v) {
  stg16_nt(p, pack16(v, static_cast<const bf16_t*>(nullptr)));
}
__device__ __forceinline__ void copy8(const float* src, float* dst) {
  stg16_nt(dst, ldg16(src));
  stg16_nt(dst + 4, ldg16(src + 4));
}
__device__ __forceinline__ void copy8(const bf16_t* src, bf16_t* dst) { stg16_nt(dst, ldg16(src)); }

// fp32(fp32(a * b) + c): multiply and add rounded separately, never fused.
__device__ __forceinline__ float mul_add_unfused(float a, float b, float c) {
#pragma clang fp contract(off)
  return a * b + c;
}

// Quantize one 8-element chunk of a fresh row and store its codes.
__device__ __forceinline__ void quantize8(const float* res, float inv, int8_t* dst) {
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    float q = rintf(__fmul_rn(res[j], inv));
    q = fminf(fmaxf(q, -127.0f), 127.0f);
    const uint32_t b = static_cast<uint32_t>(static_cast<int32_t>(q)) & 0xffu;
    w[j / 4] |= b << (8 * (j % 4));
  }
  stg8_nt(dst, make_uint2(w[0], w[1]));
}

// MAXC > 0: the fresh row's residual stays in registers (D <= 512 * MAXC);
// MAXC == 0: the row is streamed twice (any D).  FULL_ROWS (D = 512 MAXC:
// every lane owns MAXC chunks) is a kernel of its own, so that the registers
// of the ragged case do not count against it.
template <typename T, int MAXC, int CODEC, bool FULL_ROWS = false>
__global__ void __launch_bounds__(kCacheThreads)
cache_update_rows(const T* __restrict__ x, const int32_t* __restrict__ idx,
                  const uint8_t* __restrict__ mask, int n_sel, int L, int D,
                  const float* __restrict__ y_sel, T* __restrict__ xref, T* __restrict__ store,
                  int8_t* __restrict__ codes, float* __restrict__ scale, T* __restrict__ y) {
  // the value a fresh element is quantized from: its residual or itself
  auto qsrc = [](float yv, float xv) __attribute__((always_inline)) {
    return CODEC == kNaiveInt8 ? yv : __fsub_rn(yv, xv);
  };
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kCacheWavesPerBlock + wave;
  const int nch = D / 8;
  if (g < n_sel) {
    const int64_t i = idx[g];
    const float* ys = y_sel + g * D;
    const T* xi = x + i * D;
    constexpr int R = MAXC > 0 ? MAXC : 1;
    Raw8<float> yraw[R];
    Raw8<T> xraw[R];
    float amax = 0.0f;
    if (MAXC > 0) {
      // all loads of the row first; lanes past the row end re-load its last
      // chunk (in bounds) and contribute nothing
      auto body = [&](auto full_c) __attribute__((always_inline)) {
        constexpr bool FULL = decltype(full_c)::value;  // every lane owns R chunks
#pragma unroll
        for (int u = 0; u < R; ++u) {
          const int c = lane + u * kWave;
          const int cc = FULL || c < nch ? c : nch - 1;
          yraw[u].load_nt(ys + cc * 8);
          xraw[u].load_nt(xi + cc * 8);
        }
#pragma unroll
        for (int u = 0; u < R; ++u) {
          const int c = lane + u * kWave;
          if (FULL || c < nch) {
            float yv[8], xv[8];
            yraw[u].unpack(yv);
            xraw[u].unpack(xv);
            store8(y + i * D + c * 8, yv);      // fresh output, cast to storage type
            xraw[u].store_nt(xref + i * D + c * 8);  // reference := current input
            if constexpr (CODEC == kFull) {
              store8(store + i * D + c * 8, yv);
            } else {
#pragma unroll
              for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(qsrc(yv[j], xv[j])));
            }
          }
        }
      };
      body(std::integral_constant<bool, FULL_ROWS>{});
    } else if constexpr (CODEC == kFull) {
      for (int c = lane; c < nch; c += kWave) {
        float yv[8];
        load8(ys + c * 8, yv);
        store8(y + i * D + c * 8, yv);
        store8(store + i * D + c * 8, yv);
        copy8(xi + c * 8, xref + i * D + c * 8);
      }
    } else {
      for (int c = lane; c < nch; c += kWave) {
        float yv[8], xv[8];
        load8(ys + c * 8, yv);
        load8(xi + c * 8, xv);
#pragma unroll
        for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(qsrc(yv[j], xv[j])));
      }
    }
    if constexpr (CODEC == kFull) return;
    amax = wave_max(amax);
    const bool nz = amax > 0.0f;
    const float inv = nz ? __fdiv_rn(127.0f, amax) : 0.0f;
    if (lane == 0) scale[i] = nz ? __fdiv_rn(amax, 127.0f) : 0.0f;
    if (MAXC > 0) {
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        if (c < nch) {
          float yv[8], xv[8], r[8];
          yraw[u].unpack(yv);
          xraw[u].unpack(xv);
#pragma unroll
          for (int j = 0; j < 8; ++j) r[j] = qsrc(yv[j], xv[j]);  // the same values as above
          quantize8(r, inv, codes + i * D + c * 8);
        }
      }
    } else {
      for (int c = lane; c < nch; c += kWave) {
        float yv[8], xv[8], r[8];
        load8(ys + c * 8, yv);
        load8(xi + c * 8, xv);
#pragma unroll
        for (int j = 0; j < 8; ++j) r[j] = qsrc(yv[j], xv[j]);
        quantize8(r, inv, codes + i * D + c * 8);
        store8(y + i * D + c * 8, yv);
        copy8(xi + c * 8, xref + i * D + c * 8);
      }
    }
    return;
  }
  const int64_t i = g - n_sel;
  if (i >= L || mask[i]) return;
  if constexpr (CODEC == kFull) {
    if (MAXC > 0) {
      constexpr int R = MAXC > 0 ? MAXC : 1;
      Raw8<T> rr[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        if (c < nch) rr[u].load(store + i * D + c * 8);
      }
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        if (c < nch) rr[u].store_nt(y + i * D + c * 8);
      }
    } else {
      for (int c = lane; c < nch; c += kWave) copy8(store + i * D + c * 8, y + i * D + c * 8);
    }
    return;
  }
  const float sc = scale[i];
  auto reuse8 = [&](const Raw8<T>& rr, uint2 cw, int c) __attribute__((always_inline)) {
    float r[8], out[8];
    rr.unpack(r);
    const uint32_t w[2] = {cw.x, cw.y};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int8_t q = static_cast<int8_t>((w[j / 4] >> (8 * (j % 4))) & 0xffu);
      out[j] = CODEC == kNaiveInt8 ? __fmul_rn(sc, static_cast<float>(q))
                                   : mul_add_unfused(sc, static_cast<float>(q), r[j]);
    }
    store8(y + i * D + c * 8, out);
  };
  if (MAXC > 0) {
    constexpr int R = MAXC > 0 ? MAXC : 1;
    auto body = [&](auto full_c) __attribute__((always_inline)) {
      constexpr bool FULL = decltype(full_c)::value;
      Raw8<T> rr[R];
      uint2 cw[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        const int cc = FULL || c < nch ? c : nch - 1;
        if constexpr (CODEC != kNaiveInt8) rr[u].load_nt(xref + i * D + cc * 8);
        cw[u] = ldg8_nt(codes + i * D + cc * 8);
      }
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int c = lane + u * kWave;
        if (FULL || c < nch) reuse8(rr[u], cw[u], c);
      }
    };
    body(std::integral_constant<bool, FULL_ROWS>{});
  } else {
    for (int c = lane; c < nch; c += kWave) {
      Raw8<T> rr;
      if constexpr (CODEC != kNaiveInt8) rr.load(xref + i * D + c * 8);
      reuse8(rr, *reinterpret_cast<const uint2*>(codes + i * D + c * 8), c);
    }
  }
}

template <typename T, int CODEC>
static hipError_t launch_cache_t(const char* name, const T* x, const int32_t* idx, const uint8_t* mask,
                                 int n_sel, int L, int D, const float* y_sel, T* xref, T* store,
                                 int8_t* codes, float* scale, T* y, hipStream_t stream) {
  const int64_t waves = static_cast<int64_t>(n_sel) + L;
  const dim3 grid(static_cast<unsigned>((waves + kCacheWavesPerBlock - 1) / kCacheWavesPerBlock));
  const int per_lane = (D / 8 + kWave - 1) / kWave;
#define ECHO_CACHE_CASE(MC)                                                                                 \
  if (per_lane <= MC) {                                                                                     \
    if (D == 512 * MC)                                                                                      \
      return ECHO_LAUNCH(name, (cache_update_rows<T, MC, CODEC, true>), grid, dim3(kCacheThreads), 0, stream, \
                         x, idx, mask, n_sel, L, D, y_sel, xref, store, codes, scale, y);                   \
    return ECHO_LAUNCH(name, (cache_update_rows<T, MC, CODEC, false>), grid, dim3(kCacheThreads), 0, stream,  \
                       x, idx, mask, n_sel, L, D, y_sel, xref, store, codes, scale, y);                     \
  }
  ECHO_CACHE_CASE(1)
  ECHO_CACHE_CASE(2)
  ECHO_CACHE_CASE(3)
  ECHO_CACHE_CASE(4)
  ECHO_CACHE_CASE(6)
  ECHO_CACHE_CASE(8)
  ECHO_CACHE_CASE(10)
  ECHO_CACHE_CASE(12)
  ECHO_CACHE_CASE(16)
#undef ECHO_CACHE_CASE
  return ECHO_LAUNCH(name, (cache_update_rows<T, 0, CODEC>), grid, dim3(kCacheThreads), 0, stream, x, idx,
                     mask, n_sel, L, D, y_sel, xref, store, codes, scale, y);
}

template <typename T>
static hipError_t launch_codec(int codec, const T* x, const int32_t* idx, const uint8_t* mask, int n_sel,
                               int L, int D, const float* y_sel, T* xref, T* store, int8_t* codes,
                               float* scale, T* y, hipStream_t stream) {
  constexpr bool B = sizeof(T) == 2;
  switch (codec) {
    case kResidualInt8:
      return launch_cache_t<T, kResidualInt8>(B ? "cache_update_bf16" : "cache_update_f32", x, idx, mask,
                                              n_sel, L, D, y_sel, xref, store, codes, scale, y, stream);
    case kFull:
      return launch_cache_t<T, kFull>(B ? "cache_update_full_bf16" : "cache_update_full_f32", x, idx, mask,
                                      n_sel, L, D, y_sel, xref, store, codes, scale, y, stream);
    case kNaiveInt8:
      return launch_cache_t<T, kNaiveInt8>(B ? "cache_update_naive_bf16" : "cache_update_naive_f32", x, idx,
                                           mask, n_sel, L, D, y_sel, xref, store, codes, scale, y, stream);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_cache_codec(int dtype_bf16, int codec, const void* x, const int32_t* idx,
                              const uint8_t* mask, int n_sel, int L, int D, const float* y_sel, void* xref,
                              void* store, int8_t* codes, float* scale, void* y, hipStream_t stream) {
  if (dtype_bf16)
    return launch_codec<bf16_t>(codec, static_cast<const bf16_t*>(x), idx, mask, n_sel, L, D, y_sel,
                                static_cast<bf16_t*>(xref), static_cast<bf16_t*>(store), codes, scale,
                                static_cast<bf16_t*>(y), stream);
  return launch_codec<float>(codec, static_cast<const float*>(x), idx, mask, n_sel, L, D, y_sel,
                             static_cast<float*>(xref), static_cast<float*>(store), codes, scale,
                             static_cast<float*>(y), stream);
}

hipError_t launch_cache_update(int dtype_bf16, const void* x, const int32_t* idx, const uint8_t* mask,
                               int n_sel, int L, int D, const float* y_sel, void* xref, int8_t* codes,
                               float* scale, void* y, hipStream_t stream) {
  return launch_cache_codec(dtype_bf16, kResidualInt8, x, idx, mask, n_sel, L, D, y_sel, xref, nullptr, codes,
                            scale, y, stream);
}

}  // namespace echo

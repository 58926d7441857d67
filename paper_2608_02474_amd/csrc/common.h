// Shared device helpers for the gfx950 kernels: storage types, bf16 rounding,
// 16-byte vector access and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace echo {

typedef uint16_t bf16_t;                                            // storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));         // MFMA operand
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even; NaN stays NaN (quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

// Two floats rounded to bf16 (nearest even) and packed, low half first, by
// the hardware conversion (v_cvt_pk_bf16_f32): the same rounding as
// f32_to_bf16 for every non-NaN value, in one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// Element loads/stores that hide the storage type.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kPerVec = 4;  // elements per 16 bytes
  __device__ static float load(const float* p, int64_t i) { return p[i]; }
  __device__ static void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  static constexpr int kPerVec = 8;
  __device__ static float load(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  __device__ static void store(bf16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
};

// 16-byte vector of 8 bf16 or 4 fp32 unpacked to fp32.
__device__ __forceinline__ void unpack16(const uint4& v, float* out, const bf16_t*) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    out[2 * j] = __uint_as_float(w[j] << 16);
    out[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack16(const uint4& v, float* out, const float*) {
  out[0] = __uint_as_float(v.x);
  out[1] = __uint_as_float(v.y);
  out[2] = __uint_as_float(v.z);
  out[3] = __uint_as_float(v.w);
}
__device__ __forceinline__ uint4 pack16(const float* in, const bf16_t*) {
  uint4 v;
  v.x = pack_bf16x2(in[0], in[1]);
  v.y = pack_bf16x2(in[2], in[3]);
  v.z = pack_bf16x2(in[4], in[5]);
  v.w = pack_bf16x2(in[6], in[7]);
  return v;
}
__device__ __forceinline__ uint4 pack16(const float* in, const float*) {
  return make_uint4(__float_as_uint(in[0]), __float_as_uint(in[1]), __float_as_uint(in[2]),
                    __float_as_uint(in[3]));
}

__device__ __forceinline__ uint4 ldg16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}
__device__ __forceinline__ void stg16(void* p, const uint4& v) {
  *reinterpret_cast<uint4*>(p) = v;
}

// Streaming (non-temporal) 16- and 8-byte accesses, for data a kernel reads
// or writes once and that the kernels right after it do not reread.  The
// memory-bound kernels of the cached step use them for every large stream:
// measured on MI355X, the loads make the streaming kernels faster even alone,
// and the stores keep the written lines from staying dirty in the
// memory-side cache, where the next memory-bound kernel used to pay their
// write-back.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 ldg16_nt(const void* p) {
  const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ uint2 ldg8_nt(const void* p) {
  const u32x2_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  return make_uint2(t.x, t.y);
}
__device__ __forceinline__ void stg16_nt(void* p, const uint4& v) {
  const u32x4_t t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x4_t*>(p));
}
__device__ __forceinline__ void stg8_nt(void* p, const uint2& v) {
  const u32x2_t t = {v.x, v.y};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x2_t*>(p));
}

// 8 consecutive elements as raw 16-byte vectors (one for bf16, two for fp32),
// so that a row's loads can all be issued before any of them is unpacked
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> {
  uint4 v;
  __device__ void load(const bf16_t* p) { v = ldg16(p); }
  __device__ void load_nt(const bf16_t* p) { v = ldg16_nt(p); }
  __device__ void store(bf16_t* p) const { stg16(p, v); }
  __device__ void store_nt(bf16_t* p) const { stg16_nt(p, v); }
  __device__ void unpack(float* o) const { unpack16(v, o, static_cast<const bf16_t*>(nullptr)); }
};
template <> struct Raw8<float> {
  uint4 v0, v1;
  __device__ void load(const float* p) { v0 = ldg16(p); v1 = ldg16(p + 4); }
  __device__ void load_nt(const float* p) { v0 = ldg16_nt(p); v1 = ldg16_nt(p + 4); }
  __device__ void store(float* p) const { stg16(p, v0); stg16(p + 4, v1); }
  __device__ void store_nt(float* p) const { stg16_nt(p, v0); stg16_nt(p + 4, v1); }
  __device__ void unpack(float* o) const {
    unpack16(v0, o, static_cast<const float*>(nullptr));
    unpack16(v1, o + 4, static_cast<const float*>(nullptr));
  }
};

// wave64 reductions (every lane gets the result).  The partner at lane
// distance 32 and 16 comes from the gfx950 lane swaps (v_permlane32_swap,
// v_permlane16_swap: both halves of a pair in two registers), those at 8, 4,
// 2 and 1 from DPP row rotations inside the 16-lane rows, which the adder
// reads directly.  In this descending order the lane a rotation by d reaches
// holds the same value as lane i ^ d (after the steps above it, lanes that
// differ only in the bits above d's are equal), so every lane adds exactly
// the operands of an xor butterfly 32, 16, .., 1 and all lanes end with the
// same bits.  No LDS traffic: a ds_bpermute butterfly costs six LDS round
// trips per reduction.
template <int D>
__device__ __forceinline__ uint32_t dpp_ror(uint32_t v) {
  static_assert(D == 1 || D == 2 || D == 4 || D == 8, "row rotation by 1, 2, 4 or 8");
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), 0x120 + D, 0xf, 0xf, false));
}
template <typename Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = op(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = op(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  v = op(v, __uint_as_float(dpp_ror<8>(__float_as_uint(v))));
  v = op(v, __uint_as_float(dpp_ror<4>(__float_as_uint(v))));
  v = op(v, __uint_as_float(dpp_ror<2>(__float_as_uint(v))));
  v = op(v, __uint_as_float(dpp_ror<1>(__float_as_uint(v))));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ double wave_sum(double v) {
  auto swap = [](double x, auto perm) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
    const auto lo = perm(static_cast<uint32_t>(u)), hi = perm(static_cast<uint32_t>(u >> 32));
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi[0]) << 32) | lo[0])) +
           __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi[1]) << 32) | lo[1]));
  };
  v = swap(v, [](uint32_t w) { return __builtin_amdgcn_permlane32_swap(w, w, false, false); });
  v = swap(v, [](uint32_t w) { return __builtin_amdgcn_permlane16_swap(w, w, false, false); });
  auto ror = [](double x, auto d_c) {
    constexpr int D = decltype(d_c)::value;
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
    const uint64_t r = (static_cast<uint64_t>(dpp_ror<D>(static_cast<uint32_t>(u >> 32))) << 32) |
                       dpp_ror<D>(static_cast<uint32_t>(u));
    return x + __longlong_as_double(static_cast<long long>(r));
  };
  v = ror(v, std::integral_constant<int, 8>{});
  v = ror(v, std::integral_constant<int, 4>{});
  v = ror(v, std::integral_constant<int, 2>{});
  v = ror(v, std::integral_constant<int, 1>{});
  return v;
}

// Direct global-to-LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane i's bytes land at LDS offset lds_base + 16 i; lds_base is wave-uniform
// and goes through M0.  Written as inline asm on purpose: issued through the
// compiler builtin, every later LDS read of a kernel is preceded by a wait for
// ALL outstanding copies (the compiler cannot tell ring stages apart), so each
// iteration would wait for the tile it has just prefetched.  Kernels that use
// it order the copies themselves (s_waitcnt vmcnt + barrier before a stage is
// read) and use M0 for nothing else.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_copy16(const void* gsrc, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gsrc), "s"(lds_base)
               : "memory", "m0");
}
// The same copy with a wave-uniform 64-bit base in SGPRs and a 32-bit
// unsigned per-lane byte offset (the saddr form): one VGPR per copy.
__device__ __forceinline__ void lds_copy16_s(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base)
               : "memory", "m0");
}
// lds_copy16_s on the lanes of exec & exec_mask (exec_mask wave-uniform); the
// copy counts once in vmcnt whatever the lanes
__device__ __forceinline__ void lds_copy16_s_exec(const void* sbase, uint32_t voff, uint32_t lds_base,
                                                  uint64_t exec_mask) {
  uint64_t saved;
  asm volatile(
      "s_mov_b64 %0, exec\n\ts_and_b64 exec, exec, %4\n\ts_mov_b32 m0, %3\n\t"
      "global_load_lds_dwordx4 %1, %2\n\ts_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "s"(lds_base), "s"(exec_mask)
      : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt immediate (gfx9 layout) that waits until at most n vector-memory
// operations of this wave are outstanding, and for all LDS/scalar operations
// (vmcnt bits [3:0] and [15:14]; expcnt and lgkmcnt 0).
__host__ __device__ constexpr int waitcnt_vm(int n) { return (n & 15) | (((n >> 4) & 3) << 14); }

// LDS byte offset of a __shared__ object
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  // a C-style cast is the address-space conversion (generic -> LDS)
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)p));
}

}  // namespace echo

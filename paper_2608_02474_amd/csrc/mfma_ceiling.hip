// Diagnostic: the rate a dense bf16 MFMA instruction stream sustains on this
// device, by operand data.  The matrix kernels of the path are measured
// against the nominal peak (256 CUs x 4 SIMDs x 1024 bf16 FLOP per cycle at
// 2.4 GHz); the part holds that clock only while the matrix cores switch few
// bits.  With constant operands an MFMA stream runs near the nominal rate,
// with Gaussian operands (the activations and weights of the path) the clock
// falls and the same stream sustains much less.  These two kernels repeat the
// instruction patterns of the path's matrix kernels with nothing else in the
// loop (no global traffic, no barriers, no vector work), so their rate is the
// ceiling those kernels can reach on the same data:
//   * attention pattern: 12 waves (3 per SIMD), v_mfma_f32_32x32x16_bf16,
//     every MFMA takes a new A fragment from LDS (four reads in flight) and a
//     B fragment from registers, as the S and PV products of the attention;
//   * GEMM pattern: 4 waves (1 per SIMD), each an 8 x 8 grid of 16 x 16
//     accumulators, per 32-deep k step 8 A and 8 B fragments read from LDS
//     and 64 v_mfma_f32_16x16x32_bf16, the next step's fragments read during
//     the current step, as the four-wave GEMM without its copies.
// Operands: constant (1 + j/8), or Gaussian with A ~ N(0, 1) and B ~ N(0,
// 0.02) from a counter-based generator (an integer hash of the element index,
// Box-Muller), rounded to bf16.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {
namespace {

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));

// 32-bit integer hash (xorshift-multiply rounds)
__device__ __forceinline__ uint32_t hash32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return x;
}
__device__ __forceinline__ __bf16 operand(int gaussian, uint32_t key, float sigma) {
  if (!gaussian) return static_cast<__bf16>(1.0f + 0.125f * static_cast<float>(key & 7u));
  const uint32_t h = hash32(key);
  const float u1 = static_cast<float>((h >> 8) + 1u) * (1.0f / 16777217.0f);
  const float u2 = static_cast<float>(hash32(h ^ 0x9e3779b9u) >> 8) * (1.0f / 16777216.0f);
  return static_cast<__bf16>(sigma * sqrtf(-2.0f * logf(u1)) * cosf(6.2831853f * u2));
}

constexpr int kAttnWaves = 12, kGemmWaves = 4;

__global__ void __launch_bounds__(kAttnWaves * 64, 1) ceiling_attn(int gaussian, int iters, float* sink) {
  __shared__ __attribute__((aligned(1024))) __bf16 smem[32768];  // 64 KB of A fragments
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 32768; i += kAttnWaves * 64)
    smem[i] = operand(gaussian, static_cast<uint32_t>(i) * 2654435761u + blockIdx.x * 977u, 1.0f);
  __syncthreads();
  bf16x8v b[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      b[s][j] = operand(gaussian, static_cast<uint32_t>(tid * 64 + s * 8 + j) * 40503u + 7u + blockIdx.x, 0.02f);
  f32x16 c[4] = {};
  const uint32_t base = static_cast<uint32_t>(wave * 4096 + lane * 16);
  const char* sm = reinterpret_cast<const char*>(smem);
  // fragment j of pass it: 32 distinct 1 KB rows per pass, masked into the array
  auto rd = [&](int j, int it) {
    return *reinterpret_cast<const bf16x8v*>(sm + ((base + j * 1024 + (it & 1) * 32768) & 0xfff0u));
  };
  bf16x8v ring[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) ring[i] = rd(i, 0);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      c[i % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[i % 4], b[i % 8], c[i % 4], 0, 0, 0);
      ring[i % 4] = rd((i + 4) % 32, it + (i + 4) / 32);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[k][r];
  sink[blockIdx.x * blockDim.x + tid] = s;
}

__global__ void __launch_bounds__(kGemmWaves * 64, 1) ceiling_gemm(int gaussian, int iters, float* sink) {
  __shared__ __attribute__((aligned(1024))) __bf16 smem[65536];  // 64 KB of A, then 64 KB of B fragments
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 65536; i += kGemmWaves * 64)
    smem[i] = operand(gaussian, static_cast<uint32_t>(i) * 2654435761u + blockIdx.x * 977u, i < 32768 ? 1.0f : 0.02f);
  __syncthreads();
  const char* sm = reinterpret_cast<const char*>(smem);
  const uint32_t la = static_cast<uint32_t>(wave * 8192 + lane * 16);
  auto rda = [&](int j, int s) {
    return *reinterpret_cast<const bf16x8v*>(sm + ((la + j * 1024 + s * 32768) & 0xfff0u));
  };
  auto rdb = [&](int j, int s) {
    return *reinterpret_cast<const bf16x8v*>(sm + 65536 + ((la + j * 1024 + s * 32768 + 512) & 0xfff0u));
  };
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  bf16x8v fa[2][8], fb[2][8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    fa[0][j] = rda(j, 0);
    fb[0][j] = rdb(j, 0);
  }
  auto step = [&](auto set_c, int s) __attribute__((always_inline)) {
    constexpr int S = decltype(set_c)::value;
#pragma unroll
    for (int t = 0; t < 64; ++t) {
      acc[t / 8][t % 8] =
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[S][t / 8], fb[S][t % 8], acc[t / 8][t % 8], 0, 0, 0);
      if (t % 4 == 0) {
        const int q = t / 4;
        if (q < 8)
          fa[1 - S][q] = rda(q, s + 1);
        else
          fb[1 - S][q - 8] = rdb(q - 8, s + 1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  for (int it = 0; it < iters; ++it) {
    step(std::integral_constant<int, 0>{}, 2 * it);
    step(std::integral_constant<int, 1>{}, 2 * it + 1);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) s += acc[i][j][0] + acc[i][j][1] + acc[i][j][2] + acc[i][j][3];
  sink[blockIdx.x * blockDim.x + tid] = s;
}

}  // namespace

hipError_t run_mfma_ceiling(int pattern, int gaussian, double seconds, double* tflops, hipStream_t stream) {
  const int grid = 4 * device_cu_count();
  const int threads = pattern == 0 ? kAttnWaves * 64 : kGemmWaves * 64;
  // about 10 ms per launch, so that each workgroup's operand set-up (a few
  // thousand instructions per thread) stays below one percent of its time
  const int iters = pattern == 0 ? 500 : 1600;
  const double flop_per_launch = pattern == 0 ? double(grid) * kAttnWaves * iters * 32 * 32768.0
                                              : double(grid) * kGemmWaves * iters * 2 * 64 * 16384.0;
  float* sink = nullptr;
  hipError_t e = hipMallocAsync(reinterpret_cast<void**>(&sink), sizeof(float) * grid * threads, stream);
  if (e != hipSuccess) return e;
  auto launch = [&]() {
    if (pattern == 0)
      hipLaunchKernelGGL(ceiling_attn, dim3(grid), dim3(threads), 0, stream, gaussian, iters, sink);
    else
      hipLaunchKernelGGL(ceiling_gemm, dim3(grid), dim3(threads), 0, stream, gaussian, iters, sink);
    return hipGetLastError();
  };
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float ms = 0.0f;
  int reps = 0;
  if ((e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess) goto done;
  // one launch to size the run, a warm-up of about a third of the measured
  // time, then the measured launches
  if ((e = hipEventRecord(e0, stream)) != hipSuccess || (e = launch()) != hipSuccess ||
      (e = hipEventRecord(e1, stream)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess ||
      (e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess)
    goto done;
  reps = static_cast<int>(seconds * 1000.0 / (ms > 0.01f ? ms : 0.01f)) + 1;
  for (int r = 0; r < reps / 3 && e == hipSuccess; ++r) e = launch();
  if (e != hipSuccess || (e = hipEventRecord(e0, stream)) != hipSuccess) goto done;
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = launch();
  if (e != hipSuccess || (e = hipEventRecord(e1, stream)) != hipSuccess ||
      (e = hipEventSynchronize(e1)) != hipSuccess || (e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess)
    goto done;
  *tflops = flop_per_launch * reps / (double(ms) * 1e9);
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  const hipError_t ef = hipFreeAsync(sink, stream);
  return e != hipSuccess ? e : ef;
}

}  // namespace echo

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
// Tiling for gfx950: 256 x 256 output tile per 512-thread workgroup (8 waves
// as 2 x 4, each wave 128 x 64 = 4 x 2 tiles of v_mfma_f32_32x32x16_bf16),
// k-step 64, A and B tiles double-buffered in LDS (128 KB of the 160 KB), one
// barrier per k-step.  LDS rows are 128 bytes; 16-byte chunks are XOR-swizzled
// by the row index so that the 32 rows a wave reads at one k offset fall into
// distinct bank groups.  Workgroup ids are remapped so that each XCD (blocks
// are dealt round-robin to the 8 XCDs) owns a contiguous run of tiles, then
// grouped 8 tile-rows at a time so a run shares A and B panels in its L2.
// Requires N % 256 == 0 and K % 64 == 0; M is arbitrary (tail rows clamp their
// loads and skip their stores).
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int GBM = 256, GBN = 256, GBK = 64, GTHREADS = 512;

__device__ __forceinline__ int gswz(int row, int chunk) { return chunk ^ (row & 7); }

// GELU with the tanh approximation, using 0.5 z (1 + tanh u) = z / (1 + e^{-2u}).
__device__ __forceinline__ float gelu_tanh_fast(float z) {
  const float u = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z / (1.0f + __expf(-2.0f * u));
}

template <int EPI>
__global__ void __launch_bounds__(GTHREADS, 1) gemm_bf16_nt(GemmBf16Args p) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (GBM + GBN) * GBK];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave, l32 = lane & 31, hi = lane >> 5;
  const int wm = wave >> 2, wn = wave & 3;

  // ---- tile id: XCD-contiguous runs, then groups of 8 tile-rows
  const int tm = (p.M + GBM - 1) / GBM, tn = p.N / GBN, tiles = tm * tn;
  int pid = blockIdx.x;
  {
    const int q = tiles / 8, r = tiles % 8, xcd = pid % 8, loc = pid / 8;
    pid = xcd * q + (xcd < r ? xcd : r) + loc;
  }
  constexpr int GROUP = 8;
  const int group_size = GROUP * tn;
  const int first_m = (pid / group_size) * GROUP;
  const int gm = (tm - first_m) < GROUP ? (tm - first_m) : GROUP;
  const int tile_m = first_m + (pid % group_size) % gm;
  const int tile_n = (pid % group_size) / gm;
  const int m0 = tile_m * GBM, n0 = tile_n * GBN;

  // ---- per-thread global source rows and LDS destinations (4 A + 4 B chunks per k-step)
  const bf16_t* asrc[4];
  const bf16_t* bsrc[4];
  int adst[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int id = tid + GTHREADS * i;
    const int row = id >> 3, ch = id & 7;
    int m = m0 + row;
    m = m < p.M ? m : p.M - 1;
    const int64_t ar = p.a_rows ? p.a_rows[m] : m;
    asrc[i] = p.A + ar * p.lda + ch * 8;
    const int n = n0 + row;
    bsrc[i] = (n < p.n_split ? p.B0 + static_cast<int64_t>(n) * p.ldb
                             : p.B1 + static_cast<int64_t>(n - p.n_split) * p.ldb) + ch * 8;
    adst[i] = row * GBK + gswz(row, ch) * 8;
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  uint4 ra[4], rb[4];
  const int nk = p.K / GBK;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = ldg16(asrc[i]);
    rb[i] = ldg16(bsrc[i]);
  }
  {
    bf16_t* As = smem;
    bf16_t* Bs = smem + GBM * GBK;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(As + adst[i]) = ra[i];
      *reinterpret_cast<uint4*>(Bs + adst[i]) = rb[i];
    }
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      const int64_t ko = static_cast<int64_t>(kt + 1) * GBK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = ldg16(asrc[i] + ko);
        rb[i] = ldg16(bsrc[i] + ko);
      }
    }
    const bf16_t* As = smem + cur * (GBM + GBN) * GBK;
    const bf16_t* Bs = As + GBM * GBK;
#pragma unroll
    for (int s = 0; s < GBK / 16; ++s) {
      const int ch = 2 * s + hi;
      bf16x8 a[4], b[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + i * 32 + l32;
        a[i] = *reinterpret_cast<const bf16x8*>(As + row * GBK + gswz(row, ch) * 8);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wn * 64 + j * 32 + l32;
        b[j] = *reinterpret_cast<const bf16x8*>(Bs + row * GBK + gswz(row, ch) * 8);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      bf16_t* An = smem + (cur ^ 1) * (GBM + GBN) * GBK;
      bf16_t* Bn = An + GBM * GBK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<uint4*>(An + adst[i]) = ra[i];
        *reinterpret_cast<uint4*>(Bn + adst[i]) = rb[i];
      }
    }
    __syncthreads();
  }

  // ---- epilogue.  32x32 accumulator layout: lane holds column l32 and rows
  // 8*(r/4) + 4*hi + r%4 for register r.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = n0 + wn * 64 + j * 32 + l32;
    const float bias = bf16_to_f32(col < p.n_split ? p.bias0[col] : p.bias1[col - p.n_split]);
    const float gate = (EPI == EPI_GATE_RES) ? p.gate[col] : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (row >= p.M) continue;
        const float v = acc[i][j][r] + bias;
        if (EPI == EPI_BIAS) {
          static_cast<bf16_t*>(p.C)[static_cast<int64_t>(row) * p.ldc + col] = f32_to_bf16(v);
        } else if (EPI == EPI_GELU) {
          static_cast<bf16_t*>(p.C)[static_cast<int64_t>(row) * p.ldc + col] =
              f32_to_bf16(gelu_tanh_fast(v));
        } else {
          const int64_t rr = p.res_rows ? p.res_rows[row] : row;
          const float res = p.res_bf16
                                ? bf16_to_f32(static_cast<const bf16_t*>(p.res)[rr * p.ldr + col])
                                : static_cast<const float*>(p.res)[rr * p.ldr + col];
          static_cast<float*>(p.C)[static_cast<int64_t>(row) * p.ldc + col] = res + gate * v;
        }
      }
    }
  }
}

hipError_t launch_gemm_bf16(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream) {
  if (a.M <= 0) return hipSuccess;
  const int tiles = ((a.M + GBM - 1) / GBM) * (a.N / GBN);
  const dim3 grid(tiles), block(GTHREADS);
  switch (epi) {
    case EPI_BIAS:
      return ECHO_LAUNCH(name, gemm_bf16_nt<EPI_BIAS>, grid, block, 0, stream, a);
    case EPI_GELU:
      return ECHO_LAUNCH(name, gemm_bf16_nt<EPI_GELU>, grid, block, 0, stream, a);
    default:
      return ECHO_LAUNCH(name, gemm_bf16_nt<EPI_GATE_RES>, grid, block, 0, stream, a);
  }
}

}  // namespace echo

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
// Tiling for gfx950: 256 x 256 output tiles, one workgroup of four waves
// (one per SIMD) per tile, each wave a 128 x 128 quarter as 8 x 8 blocks of
// v_mfma_f32_16x16x32_bf16, k-steps of 64 through a two-stage LDS ring that
// direct global-to-LDS copies fill (gemm_bf16_w4 below).
// Tiles are taken in a grouped order (8 tile-rows at a time, down the rows
// first) and dealt so that the tiles running together on the 8 XCDs (blocks
// go round-robin to the XCDs) form one block of 8 tile-rows: every L2 works
// on the same A panels at the same time, so that the misses of one L2 find
// what another has just brought into the memory-side cache instead of going
// to HBM (the L2s miss as often either way: about five times the algorithmic
// bytes on the K/V shape).  Tiles that do not fill a
// last round of the device are split along k, run first in the same launch
// (gemm_splitk_reduce adds the ranges in order and applies the epilogue).
// Requires N % BN == 0, n_split % BN == 0, K % BK == 0 and byte offsets of
// A and B rows below 2^31; M is arbitrary (tail rows clamp their loads and
// skip their stores).
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// GELU with the tanh approximation, using 0.5 z (1 + tanh u) = z / (1 + e^{-2u})
// with u = sqrt(2/pi) (z + 0.044715 z^3): e^{-2u} = 2^{z (k1 + k2 z^2)}, k1 =
// -2 sqrt(2/pi) log2(e), k2 = 0.044715 k1, so the argument is one FMA and two
// products (the unfolded form took six products, an FMA and an add per
// element).  exp2 and the reciprocal are the hardware ones (1 ulp), far below
// the bf16 rounding of the result; z -> -inf gives z * 0, z -> +inf gives z.
__device__ __forceinline__ float gelu_tanh_fast(float z) {
  constexpr double kU = 0.7978845608028654 * 1.4426950408889634;  // sqrt(2/pi) log2(e)
  constexpr float k1 = static_cast<float>(-2.0 * kU), k2 = static_cast<float>(-2.0 * kU * 0.044715);
  const float e = __builtin_amdgcn_exp2f(z * fmaf(k2, z * z, k1));
  return z * __builtin_amdgcn_rcpf(1.0f + e);
}

// Grouped tile order: 8 tile-rows at a time, down the rows first, so that
// consecutive tiles share B panels and a run of them shares A panels in L2.
__host__ __device__ __forceinline__ void gemm_tile_of(int pid, int tm, int tn, int& tile_m, int& tile_n) {
  constexpr int GROUP = 8;
  const int group_size = GROUP * tn;
  const int first_m = (pid / group_size) * GROUP;
  const int gm = (tm - first_m) < GROUP ? (tm - first_m) : GROUP;
  tile_m = first_m + (pid % group_size) % gm;
  tile_n = (pid % group_size) / gm;
}

// Bias (and gate) of the 4 consecutive output columns col .. col+3.
template <int EPI>
__device__ __forceinline__ void gemm_col4(const GemmBf16Args& p, int col, float* bias, float* gate) {
  const bf16_t* bias_p = col < p.n_split ? p.bias0 + col : p.bias1 + (col - p.n_split);
  const uint2 bb = *reinterpret_cast<const uint2*>(bias_p);
  bias[0] = __uint_as_float(bb.x << 16);
  bias[1] = __uint_as_float(bb.x & 0xffff0000u);
  bias[2] = __uint_as_float(bb.y << 16);
  bias[3] = __uint_as_float(bb.y & 0xffff0000u);
  if (EPI == EPI_GATE_RES) {
    const float4 g = *reinterpret_cast<const float4*>(p.gate + col);
    gate[0] = g.x; gate[1] = g.y; gate[2] = g.z; gate[3] = g.w;
  }
}

// Residual of the 4 consecutive columns col .. col+3 of row `row` (gathered
// through res_rows if given), bf16 or fp32, as fp32.
__device__ __forceinline__ void gemm_res4(const GemmBf16Args& p, int row, int col, float* res) {
  const int64_t rr = p.res_rows ? p.res_rows[row] : row;
  if (p.res_bf16) {
    const uint2 rb = ldg8_nt(static_cast<const bf16_t*>(p.res) + rr * p.ldr + col);
    res[0] = __uint_as_float(rb.x << 16);
    res[1] = __uint_as_float(rb.x & 0xffff0000u);
    res[2] = __uint_as_float(rb.y << 16);
    res[3] = __uint_as_float(rb.y & 0xffff0000u);
  } else {
    const uint4 rf = ldg16_nt(static_cast<const float*>(p.res) + rr * p.ldr + col);
    res[0] = __uint_as_float(rf.x); res[1] = __uint_as_float(rf.y); res[2] = __uint_as_float(rf.z); res[3] = __uint_as_float(rf.w);
  }
}

// Output of 4 consecutive columns col .. col+3 of row `row` (acc4 = sums
// without bias; res = the residual of those columns for EPI_GATE_RES).  The
// fp32 gate + residual outputs and their residual reads are streams read or
// written once, so they use the non-temporal accesses (O projection
// 0.687 -> 0.653 ms, FFN down 1.657 -> 1.645 ms); the bf16 outputs are read
// by the next kernel and keep ordinary stores.
template <int EPI>
__device__ __forceinline__ void gemm_store4(const GemmBf16Args& p, int row, int col, const float* acc4,
                                            const float* bias, const float* gate, const float* res) {
  float v[4] = {acc4[0] + bias[0], acc4[1] + bias[1], acc4[2] + bias[2], acc4[3] + bias[3]};
  if (EPI == EPI_GATE_RES) {
    float4 o;
    o.x = res[0] + gate[0] * v[0];
    o.y = res[1] + gate[1] * v[1];
    o.z = res[2] + gate[2] * v[2];
    o.w = res[3] + gate[3] * v[3];
    stg16_nt(static_cast<float*>(p.C) + static_cast<int64_t>(row) * p.ldc + col, make_uint4(__float_as_uint(o.x), __float_as_uint(o.y), __float_as_uint(o.z), __float_as_uint(o.w)));
  } else {
    if (EPI == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = gelu_tanh_fast(v[e]);
    }
    uint2 o;
    o.x = pack_bf16x2(v[0], v[1]);
    o.y = pack_bf16x2(v[2], v[3]);
    *reinterpret_cast<uint2*>(static_cast<bf16_t*>(p.C) + static_cast<int64_t>(row) * p.ldc + col) = o;
  }
}

// ---- the tile kernel.  Each wave owns a 128 x 128 quarter of the tile as
// 8 x 8 blocks of v_mfma_f32_16x16x32_bf16 (accumulators: 256 AGPRs per lane;
// fragments of two k32 halves in flight: 128 VGPRs).  The LDS holds two
// stages of 64 KB (A ++ B, 512 rows of 128 bytes; the 16-byte chunk of row r
// is XOR-swizzled by (r >> 1) & 7, so that the 16 rows one LDS cycle serves
// hit 16 distinct bank groups).  A k-step is
//   (0)  the 64 MFMAs of its first k32 half, with the 16 fragment reads of
//        the second half and the last 8 copies of the k-step after next
//        between them (one read per four MFMAs, one copy per four MFMAs over
//        the first 32);
//   (1a) 32 MFMAs of the second half;
//   --   a wait for this wave's copies of the next k-step and a barrier:
//        after it the next stage is complete everywhere and no wave reads
//        the current one any more (its fragments are all in registers);
//   (1b) the last 32 MFMAs, with the 16 reads of the next k-step's first half
//        and the first 8 copies of the k-step after next into the stage just
//        released.
// A copy thus has about one k-step to land, and a k-step's only wait sits
// between MFMAs.  The loop runs from one barrier to the next ((1b) of k-step
// kt, then (0) and (1a) of kt + 1), so every fragment read is used in the
// iteration that issues it and the compiler's wait counts stay exact.  Past
// the last k-step the copies re-fetch it (in bounds, never read).  Against
// the earlier 8-wave form (32x32x16 MFMAs, 128 x 64 per wave, a four-stage
// ring of k32 steps) this reads a third fewer LDS bytes per MFMA and keeps
// the MFMA pipes busier: K/V projection 2.90 -> 2.46 ms, FFN 1.66 -> 1.45 ms.
constexpr int kW4Threads = 256;
constexpr int kW4Stage = 512 * 128;
// copy and barrier placement (measured: 8 / 8 / 32 beat 16 / -, 10 / 6, 6 / 8,
// 4 / 6, 8 / 4 and 8 / 16 copies, and 24 or 40 MFMAs before the barrier)
constexpr int kW4CopiesIn1b = 8;     // copies issued in (1b); the rest in (0)
constexpr int kW4CopyGroups0 = 8;    // the first groups of (0) that carry them
constexpr int kW4Mfma1a = 32;        // MFMAs of the second half before the barrier

template <int EPI>
__global__ void __launch_bounds__(kW4Threads, 1) gemm_bf16_w4(GemmBf16Args p) {
  constexpr int BM = 256, BN = 256, BK = 64;
  __shared__ __attribute__((aligned(1024))) char smem[2 * kW4Stage];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, lq = lane >> 4;

  // ---- tile id.  Workgroups g < npieces are k-split pieces: k-range
  // g % nsplit of tile tile_base + g / nsplit.  The rest take whole tiles
  // [0, gridDim.x - npieces) of the grouped order, dealt to the XCDs as below.
  const int tm = (p.M + BM - 1) / BM, tn = p.N / BN;
  const bool split_k = static_cast<int>(blockIdx.x) < p.npieces;
  int pid, ksplit = 0;
  if (!split_k) {
    // workgroup g runs on XCD g % 8 as that XCD's (g / 8)-th; the XCDs'
    // workgroups loc 32 w .. 32 w + 31 run together, so tile wave w of all
    // eight XCDs takes grouped tiles 256 w .. 256 w + 255 (8 tile-rows x 32
    // tile-columns), XCD x the 32 from 256 w + 32 x: the eight L2s work on
    // the same A panels at the same time (shared through the memory-side
    // cache) instead of each streaming its own; a last partial wave keeps the
    // identity order
    const int g = blockIdx.x - p.npieces, xcd = g % 8, loc = g / 8;
    const int full_waves = (gridDim.x - p.npieces) / 256;
    pid = loc < 32 * full_waves ? (loc / 32) * 256 + xcd * 32 + loc % 32 : g;
  } else {
    pid = p.tile_base + blockIdx.x / p.nsplit;
    ksplit = blockIdx.x % p.nsplit;
  }
  int tile_m, tile_n;
  gemm_tile_of(pid, tm, tn, tile_m, tile_n);
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // ---- copy plan: copy c of this wave fills the 8 rows 8 (wave + 4 c) ..
  // of the (A ++ B) stage, c < 8 in A; lane i takes row + i / 8, slot i % 8,
  // which holds logical chunk (i % 8) ^ ((row >> 1) & 7)
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const bf16_t* b_base = n0 < p.n_split ? p.B0 : p.B1;  // BN divides n_split
  const int n_off = n0 < p.n_split ? n0 : n0 - p.n_split;
  // The swizzled chunk of a lane, (lane % 8) ^ ((row >> 1) & 7), is the same
  // for all its copies (rows 32 apart).  A rows may be gathered, so each A copy
  // keeps its own offset; the B copies are one offset plus 32 rows per copy,
  // folded into the wave-uniform base.
  const int chunk = (lane % 8) ^ (((8 * wave_u + lane / 8) >> 1) & 7);
  uint32_t voff_a[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    int m = m0 + 8 * (wave_u + 4 * c) + lane / 8;
    m = m < p.M ? m : p.M - 1;
    const uint32_t ar = p.a_rows ? static_cast<uint32_t>(p.a_rows[m]) : static_cast<uint32_t>(m);
    voff_a[c] = (ar * static_cast<uint32_t>(p.lda) + chunk * 8) * 2u;
  }
  const uint32_t voff_b =
      ((n_off + 8 * wave_u + lane / 8) * static_cast<uint32_t>(p.ldb) + chunk * 8) * 2u;
  const int64_t b_copy_step = 32 * p.ldb;  // elements between consecutive B copies
  const uint32_t dst0 = lds_offset(smem) + wave_u * 1024;  // copy c lands at dst0 + 4096 c
  const int nk_all = p.K / BK;
  const int kt0 = split_k ? ksplit * p.kps : 0;
  const int nk = split_k ? (nk_all - kt0 < p.kps ? nk_all - kt0 : p.kps) : nk_all;  // >= 1
  const bf16_t* src_a = p.A;
  const bf16_t* src_b = b_base;
  uint32_t dst_stage = 0;
  auto set_fill = [&](int kt, int stage) __attribute__((always_inline)) {
    const int kf = kt0 + (kt < nk ? kt : nk - 1);
    src_a = p.A + static_cast<int64_t>(kf) * BK;
    src_b = b_base + static_cast<int64_t>(kf) * BK;
    dst_stage = dst0 + stage * kW4Stage;
  };
  auto copy = [&](auto c_c) __attribute__((always_inline)) {
    constexpr int c = decltype(c_c)::value;
    if constexpr (c < 8)
      lds_copy16_s(src_a, voff_a[c], dst_stage + c * 4096);
    else
      lds_copy16_s(src_b + (c - 8) * b_copy_step, voff_b, dst_stage + c * 4096);
  };

  // ---- fragments: read q (0..15) of a k32 half is A block 0, then B blocks
  // 0..7, then A blocks 1..7, the order the MFMAs (A block outer) use them
  const int rd_a = (wm * 128 + l16) * 128, rd_b = (BM + wn * 128 + l16) * 128;
  const int ch0 = (lq ^ (l16 >> 1)) * 16, ch1 = ((4 + lq) ^ (l16 >> 1)) * 16;
  bf16x8 fa[2][8], fb[2][8];
  auto read = [&](auto set_c, auto q_c, const char* base, int half) __attribute__((always_inline)) {
    constexpr int SET = decltype(set_c)::value, Q = decltype(q_c)::value;
    const int ch = half ? ch1 : ch0;
    if constexpr (Q == 0)
      fa[SET][0] = *reinterpret_cast<const bf16x8*>(base + rd_a + ch);
    else if constexpr (Q <= 8)
      fb[SET][Q - 1] = *reinterpret_cast<const bf16x8*>(base + rd_b + (Q - 1) * 2048 + ch);
    else
      fa[SET][Q - 8] = *reinterpret_cast<const bf16x8*>(base + rd_a + (Q - 8) * 2048 + ch);
  };
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  auto mma = [&](auto set_c, auto t0_c, auto t1_c) __attribute__((always_inline)) {
    constexpr int SET = decltype(set_c)::value, T0 = decltype(t0_c)::value, T1 = decltype(t1_c)::value;
    static_for<T0, T1>([&](auto t_c) __attribute__((always_inline)) {
      constexpr int T = decltype(t_c)::value;
      acc[T / 8][T % 8] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[SET][T / 8], fb[SET][T % 8],
                                                                  acc[T / 8][T % 8], 0, 0, 0);
    });
  };
  typedef std::integral_constant<int, 0> S0;
  typedef std::integral_constant<int, 1> S1;

  // ---- prologue: k-steps 0 and 1 (or k-step 0 again) in flight, k-step 0
  // complete; the MFMAs of k-step 0 up to the first barrier
  set_fill(0, 0);
  static_for<0, 16>(copy);
  set_fill(1, 1);
  static_for<0, 16>(copy);
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(16));
  __syncthreads();
  static_for<0, 16>([&](auto q_c) __attribute__((always_inline)) { read(S0{}, q_c, smem, 0); });
  // (0) of a k-step: the first half's 64 MFMAs with the second half's reads
  // (and the copies that (1b) left, CS .. 15)
  auto phase0 = [&](const char* stage, auto cs_c) __attribute__((always_inline)) {
    constexpr int CS = decltype(cs_c)::value;
    static_for<0, 16>([&](auto q_c) __attribute__((always_inline)) {
      constexpr int Q = decltype(q_c)::value;
      __builtin_amdgcn_sched_barrier(0);
      mma(S0{}, std::integral_constant<int, 4 * Q>{}, std::integral_constant<int, 4 * Q + 4>{});
      read(S1{}, q_c, stage, 1);
      // the copies CS .. 15 spread evenly over the first P0 groups
      constexpr int NC = 16 - CS, P0 = kW4CopyGroups0;
      if constexpr (Q < P0) static_for<CS + Q * NC / P0, CS + (Q + 1) * NC / P0>(copy);
    });
    __builtin_amdgcn_sched_barrier(0);
  };
  typedef std::integral_constant<int, 16> NoCopies;
  constexpr int H1A = kW4Mfma1a;  // MFMAs of the second half before the barrier
  typedef std::integral_constant<int, kW4CopiesIn1b> Cs;
  phase0(smem, NoCopies{});
  mma(S1{}, std::integral_constant<int, 0>{}, std::integral_constant<int, H1A>{});  // (1a)
  __builtin_amdgcn_sched_barrier(0);
  // One iteration: the barrier of k-step kt, its last 32 MFMAs (1b) with the
  // first-half reads of kt + 1 and the first copies of kt + 2, then (0) and
  // (1a) of kt + 1.  The reads of an iteration are used in that iteration.
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const char* nxt = smem + ((kt & 1) ^ 1) * kW4Stage;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // this wave's copies of k-step kt + 1
    __syncthreads();
    set_fill(kt + 2, kt & 1);
    static_for<0, 16>([&](auto q_c) __attribute__((always_inline)) {
      constexpr int Q = decltype(q_c)::value;
      constexpr int M1 = 64 - H1A;  // MFMAs of (1b), spread over its 16 reads
      __builtin_amdgcn_sched_barrier(0);
      mma(S1{}, std::integral_constant<int, H1A + Q * M1 / 16>{},
          std::integral_constant<int, H1A + (Q + 1) * M1 / 16>{});
      read(S0{}, q_c, nxt, 0);
      static_for<Q * Cs::value / 16, (Q + 1) * Cs::value / 16>(copy);
    });
    __builtin_amdgcn_sched_barrier(0);
    phase0(nxt, Cs{});
    mma(S1{}, std::integral_constant<int, 0>{}, std::integral_constant<int, H1A>{});  // (1a)
    __builtin_amdgcn_sched_barrier(0);
  }
  mma(S1{}, std::integral_constant<int, H1A>{}, std::integral_constant<int, 64>{});  // (1b) of the last k-step
  __builtin_amdgcn_s_waitcnt(0);  // re-fetched k-steps still landing in LDS
  __syncthreads();

  // ---- epilogue: each wave stages one 16-row group of its quarter at a time
  // (lane holds column l16 and rows 4 lq .. 4 lq + 3 of every block) and reads
  // it back as 4 consecutive columns per lane, two rows per read.  Rows are
  // padded by 4 floats, so the four row groups of a write hit distinct banks.
  constexpr int EP_LD = 128 + 4;
  float* ep = reinterpret_cast<float*>(smem) + wave * 16 * EP_LD;
  const int c_l = (lane % 32) * 4;
  const int col = n0 + wn * 128 + c_l;
  float bias[4], gate[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (!split_k) gemm_col4<EPI>(p, col, bias, gate);
  constexpr int NR = EPI == EPI_GATE_RES ? 8 : 1;
  // Gate + residual: the residual rows of group i are the lane's rows
  // m0 + wm 128 + 16 i + 2 q + lane / 32 (q < 8), gathered through res_rows
  // if given.  bf16 residuals (the O projection's gathered block input) are
  // fetched NPF = 2 groups ahead, their row indices three groups ahead, so
  // that the latency hides behind the staging and stores of the groups
  // before (O projection: no prefetch 0.599 ms, one group 0.583 - 0.600, two
  // groups 8 us less, three or four no better); fp32 residuals (read once, no
  // gather) are fetched at the start of their group, where the prefetch
  // gained nothing and cost registers.
  constexpr bool RES = EPI == EPI_GATE_RES;
  constexpr int NQ = RES ? 8 : 1;
  const bool pre = RES && !split_k && p.res_bf16;
  constexpr int NPF = 2, NS = NPF + 1;
  int32_t rrow[2][NQ];  // row indices of groups g in slot g % 2
  uint2 rawb[NS][NQ];   // residuals of group g in slot g % NS
  auto rows_of = [&](int i, int32_t(&dst)[NQ]) __attribute__((always_inline)) {
    if constexpr (RES) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int row = m0 + wm * 128 + i * 16 + 2 * q + lane / 32;
        dst[q] = row < p.M ? row : p.M - 1;
      }
      if (p.res_rows != nullptr) {
#pragma unroll
        for (int q = 0; q < 8; ++q) dst[q] = p.res_rows[dst[q]];
      }
    }
  };
  auto load_bf16 = [&](const int32_t(&rr)[NQ], uint2(&dst)[NQ]) __attribute__((always_inline)) {
    if constexpr (RES) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        dst[q] = ldg8_nt(static_cast<const bf16_t*>(p.res) + static_cast<int64_t>(rr[q]) * p.ldr + col);
    }
  };
  if (pre) {
#pragma unroll
    for (int g = 0; g < NPF; ++g) {
      rows_of(g, rrow[g % 2]);
      load_bf16(rrow[g % 2], rawb[g]);
    }
    rows_of(NPF, rrow[NPF % 2]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float res[NR][4];
    if constexpr (RES) {
      if (pre) {
        // issue the residuals of group i + NPF (its rows are in slot
        // (i + NPF) % 2), then fetch the rows of group i + NPF + 1 into the
        // other slot, whose group's residuals were issued the group before
        if (i + NPF < 8) load_bf16(rrow[(i + NPF) % 2], rawb[(i + NPF) % NS]);
        if (i + NPF + 1 < 8) rows_of(i + NPF + 1, rrow[(i + NPF + 1) % 2]);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint2 v = rawb[i % NS][q];
          res[q][0] = __uint_as_float(v.x << 16);
          res[q][1] = __uint_as_float(v.x & 0xffff0000u);
          res[q][2] = __uint_as_float(v.y << 16);
          res[q][3] = __uint_as_float(v.y & 0xffff0000u);
        }
      } else if (!split_k) {
        int32_t rr[8];
        rows_of(i, rr);
        const float* rf = static_cast<const float*>(p.res) + col;
        uint4 raw[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) raw[q] = ldg16_nt(rf + static_cast<int64_t>(rr[q]) * p.ldr);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          res[q][0] = __uint_as_float(raw[q].x);
          res[q][1] = __uint_as_float(raw[q].y);
          res[q][2] = __uint_as_float(raw[q].z);
          res[q][3] = __uint_as_float(raw[q].w);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) ep[(4 * lq + r) * EP_LD + j * 16 + l16] = acc[i][j][r];
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(63));  // this wave's staged group is in LDS
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r_l = 2 * q + lane / 32;
      const int trow = wm * 128 + i * 16 + r_l;
      const float4 a4 = *reinterpret_cast<const float4*>(ep + r_l * EP_LD + c_l);
      if (split_k) {
        *reinterpret_cast<float4*>(p.part + static_cast<int64_t>(blockIdx.x) * BM * BN +
                                   static_cast<int64_t>(trow) * BN + (col - n0)) = a4;
      } else if (m0 + trow < p.M) {
        const float v[4] = {a4.x, a4.y, a4.z, a4.w};
        gemm_store4<EPI>(p, m0 + trow, col, v, bias, gate, res[EPI == EPI_GATE_RES ? q : 0]);
      }
    }
  }
}

// Sum the k-range partials of the split tail tiles in split order and apply
// the epilogue.  One thread per 4 output columns.
template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(256) gemm_splitk_reduce(GemmBf16Args p, int ntail) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(ntail) * BM * (BN / 4)) return;
  const int c4 = static_cast<int>(e % (BN / 4)), trow = static_cast<int>((e / (BN / 4)) % BM);
  const int j = static_cast<int>(e / (static_cast<int64_t>(BM) * (BN / 4)));
  const int tm = (p.M + BM - 1) / BM, tn = p.N / BN;
  int tile_m, tile_n;
  gemm_tile_of(p.tile_base + j, tm, tn, tile_m, tile_n);
  const int row = tile_m * BM + trow;
  if (row >= p.M) return;
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int sp = 0; sp < p.nsplit; ++sp) {
    const float4 a4 = *reinterpret_cast<const float4*>(
        p.part + (static_cast<int64_t>(j) * p.nsplit + sp) * BM * BN + static_cast<int64_t>(trow) * BN + 4 * c4);
    v[0] += a4.x;
    v[1] += a4.y;
    v[2] += a4.z;
    v[3] += a4.w;
  }
  float bias[4], gate[4] = {0.0f, 0.0f, 0.0f, 0.0f}, res[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  gemm_col4<EPI>(p, tile_n * BN + 4 * c4, bias, gate);
  if (EPI == EPI_GATE_RES) gemm_res4(p, row, tile_n * BN + 4 * c4, res);
  gemm_store4<EPI>(p, row, tile_n * BN + 4 * c4, v, bias, gate, res);
}

// The tile kernel the launcher runs.
template <int EPI>
struct GemmW4 {
  static constexpr int kThreads = kW4Threads;
  static void launch(int grid, const GemmBf16Args& a, hipStream_t stream) {
    hipLaunchKernelGGL((gemm_bf16_w4<EPI>), dim3(grid), dim3(kThreads), 0, stream, a);
  }
};

template <int BM, int BN, int BK, int EPI, typename KERNEL>
hipError_t launch_gemm_epi(const char* name, GemmBf16Args a, hipStream_t stream) {
  const int tiles = ((a.M + BM - 1) / BM) * (a.N / BN);
  const int nk = a.K / BK;
  // Tiles beyond the last full round (one workgroup per CU) are split along
  // k; a reduce kernel adds the splits.  A tail of at least a quarter of the
  // CUs is cut so that its pieces fill that round; a smaller one into about
  // 3/16 of the CUs' worth of pieces (with 256 CUs, measured in the cached
  // block step: 64 tail tiles in 4 pieces each beat 3, 2 and 1; 16 tiles in
  // 3 beat 2, 4 and 8 (O projection 562 -> 545 us, FFN down 1377 -> 1331
  // us); 8 tiles in 6 beat 4 and 8; 4 tiles in the 8 that the k-step floor
  // below allows beat 6, 4 and 3).
  const int ncu = device_cu_count();
  const int tail = tiles % ncu;
  int nsplit = 1;
  if (tail > 0) nsplit = 4 * tail >= ncu ? ncu / tail : (3 * ncu / 16 + tail - 1) / tail;
  nsplit = nsplit < nk ? nsplit : nk;
  // Each split also writes and the reduce reads a 256 KB fp32 partial tile:
  // below about 640 of depth (10 k-steps) per split that costs more than the
  // shorter range saves.
  constexpr int kMinStepsPerSplit = 640 / BK;
  const int cap = nk / kMinStepsPerSplit > 1 ? nk / kMinStepsPerSplit : 1;
  nsplit = nsplit < cap ? nsplit : cap;
  const size_t unit_bytes = sizeof(float) * BM * BN;
  while (nsplit > 1 && static_cast<size_t>(tail) * nsplit * unit_bytes > a.part_bytes) --nsplit;
  if (a.part == nullptr) nsplit = 1;
  ::echo::TimedLaunch scope(name, stream);
  a.tile_base = 0;
  a.npieces = 0;
  if (nsplit < 2) {
    a.nsplit = 1;
    KERNEL::launch(tiles, a, stream);
    return hipGetLastError();
  }
  a.kps = (nk + nsplit - 1) / nsplit;  // k-steps per split
  nsplit = (nk + a.kps - 1) / a.kps;   // every split non-empty
  // One launch, the pieces first: when they cover only part of the CUs (the
  // 13104-row projections: 16 tiles x 3 pieces), the other CUs start on whole
  // tiles and stay a piece's time ahead, so that the rounds' epilogues no
  // longer store at the same moment on every CU (O projection with 8 pieces a
  // tile: 577 -> 563 us against whole tiles first, then the pieces, in two
  // launches).
  const int full = tiles - tail;
  a.tile_base = full;
  a.nsplit = nsplit;
  a.npieces = tail * nsplit;
  KERNEL::launch(tail * nsplit + full, a, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t threads = static_cast<int64_t>(tail) * BM * (BN / 4);
  hipLaunchKernelGGL((gemm_splitk_reduce<BM, BN, EPI>), dim3(static_cast<unsigned>((threads + 255) / 256)),
                     dim3(256), 0, stream, a, tail);
  return hipGetLastError();
}

hipError_t launch_gemm_w4(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream) {
  constexpr int BM = 256, BN = 256, BK = 64;
  if (a.N % BN != 0 || (a.n_split < a.N && a.n_split % BN != 0) || a.K % BK != 0)
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_BIAS: return launch_gemm_epi<BM, BN, BK, EPI_BIAS, GemmW4<EPI_BIAS>>(name, a, stream);
    case EPI_GELU: return launch_gemm_epi<BM, BN, BK, EPI_GELU, GemmW4<EPI_GELU>>(name, a, stream);
    default: return launch_gemm_epi<BM, BN, BK, EPI_GATE_RES, GemmW4<EPI_GATE_RES>>(name, a, stream);
  }
}

hipError_t launch_gemm_bf16(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream) {
  if (a.M <= 0) return hipSuccess;
  // the tile loads address A and B through 32-bit byte offsets
  const int64_t lim = int64_t(1) << 31;
  if (a.a_nrows <= 0 || a.a_nrows * a.lda * 2 >= lim || int64_t(a.N) * a.ldb * 2 >= lim)
    return hipErrorInvalidValue;
  return launch_gemm_w4(name, epi, a, stream);
}

}  // namespace echo

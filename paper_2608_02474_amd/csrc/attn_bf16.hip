// Restricted-query attention (Sec. 3.3, "Fine-grained latent-level caching"):
// the queries of the selected tokens attend over the keys and values of ALL
// tokens, per head, o = softmax(q k^T / sqrt(dh)) v, dh = 128, bf16 operands
// with fp32 accumulation and an online (streaming) softmax.
//
// gfx950 mapping.  A workgroup of WAVES waves owns WAVES * QB * 32 queries of
// one head (each wave QB blocks of 32 queries).  Keys stream in tiles of 64:
//   * K and V tiles are copied HBM/L2 -> LDS by direct global-to-LDS loads
//     (global_load_lds_dwordx4: no VGPR staging), row-major [key][dh], into a
//     3-stage ring.  Each lane fetches the 16-byte piece whose swizzled LDS
//     slot is its own lane slot, so the XOR swizzles cost nothing at load time.
//   * S^T (keys x queries) = K_tile . Q^T with v_mfma_f32_32x32x16_bf16; the
//     query fragments stay in registers for the whole key loop; K rows enter
//     the MFMA in a permuted order (bits 2 and 3 of the row index swapped) so
//     that each lane's accumulators hold 8 consecutive keys per 16-key step.
//   * S of tile t+1 is issued before the softmax of tile t, so the MFMA pipe
//     works while the VALU runs exp/max/sum of the previous tile.
//   * softmax per lane: a lane owns one query per block (its accumulator
//     column) and half of the tile's keys; the row max uses one
//     v_permlane32_swap.  The scale is folded into one FMA before exp2;
//     masking runs only on the ragged last tile; a row's running output is
//     rescaled only when the tile raises its maximum by more than 2^8 (rows
//     that keep their maximum are untouched, so each row's arithmetic depends
//     on its own scores only).
//   * O^T (dh x queries) += V^T . P^T: P^T is the S accumulator converted to
//     bf16 in registers; V^T fragments come straight from the row-major V tile
//     with ds_read_b64_tr_b16 (LDS transpose reads), two per 8-key operand.
// Workgroup ids are remapped so that each XCD works through a contiguous range
// of (head, query-tile) pairs: the query tiles of one head share that head's
// K/V stream in one L2.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int ATT_KT = 64, ATT_DH = 128;
constexpr int ATT_TILE_BYTES = ATT_KT * ATT_DH * 2;  // one K or V tile: 16 KB
constexpr int ATT_STAGE_BYTES = 2 * ATT_TILE_BYTES;  // K + V
constexpr int ATT_OS_STRIDE = ATT_DH + 8;            // output staging row (bf16)
constexpr float ATT_RESCALE_LOG2 = 8.0f;             // lazy-rescale headroom (log2 units)

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// MODE 0: per tile, barrier -> S -> softmax -> PV.
// MODE 1: S of the next tile issued before the softmax of this one.
// MODE 2: ping-pong.  The waves split into two groups that run the same
//         two-phase loop (phase A: PV of the previous tile + S of this tile on
//         the MFMA pipe; phase B: softmax on the VALU) one phase apart, so on
//         every SIMD one wave feeds the matrix pipe while the other runs exp.
template <int QB, int WAVES, int MODE>
struct AttCfg {
  static constexpr int kThreads = WAVES * 64;
  static constexpr int kQ = WAVES * QB * 32;  // queries per workgroup
  static constexpr int kStages = MODE == 2 ? 4 : 3;
  static constexpr int kLdsBytes = (kStages * ATT_STAGE_BYTES > kQ * ATT_OS_STRIDE * 2)
                                       ? kStages * ATT_STAGE_BYTES
                                       : kQ * ATT_OS_STRIDE * 2;
};

// swap bits 2 and 3
__device__ __forceinline__ int perm23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// K tile row r (256 B = 16 chunks of 16 B): logical chunk c lives in slot c ^ perm23(r & 15).
// Lanes reading rows perm23(l) at one chunk then hit 8 distinct 16-byte bank groups.
__device__ __forceinline__ int k_slot(int r, int c) { return c ^ perm23(r & 15); }
// V tile row r (256 B = 8 blocks of 32 B): logical block b lives in block
// b ^ 2(r & 3).  One half-wave of a transpose read (the 256 B one LDS cycle
// serves) touches 4 consecutive rows of the logical blocks 2d and 2d+1; these
// 8 pieces land in the 8 distinct physical blocks.
__device__ __forceinline__ int v_block(int r, int b) { return b ^ ((r & 3) << 1); }

__device__ __forceinline__ float pair_max(float x) {
  // max over lanes l and l^32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

#define ECHO_LDS(p) ((__attribute__((address_space(3))) void*)(p))

#define ECHO_LDS_V4(p) ((__attribute__((address_space(3))) v4i16*)(p))

template <int QB, int WAVES, int MODE>
__global__ void __launch_bounds__(WAVES * 64, 1)
attn_fwd_bf16(const bf16_t* __restrict__ q, int64_t ldq, const bf16_t* __restrict__ k,
              const bf16_t* __restrict__ v, int64_t ldkv, int Mq, int L, int H, float scale_log2,
              bf16_t* __restrict__ out, int64_t ldo) {
  typedef AttCfg<QB, WAVES, MODE> C;
  constexpr int ATT_NSTAGE = C::kStages;
  constexpr int NLD = 16 / WAVES;  // 1 KB direct-load instructions per wave per K (or V) tile
  static_assert(16 % WAVES == 0, "16 KB tiles split evenly over the waves");
  __shared__ __attribute__((aligned(1024))) char smem[C::kLdsBytes];

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave, l32 = lane & 31, hi = lane >> 5;
  const int g16 = lane >> 4, i16 = lane & 15;

  const int ntq = (Mq + C::kQ - 1) / C::kQ;
  const int total = ntq * H;
  int pid = blockIdx.x;
  {
    const int qq = total / 8, r = total % 8, xcd = pid % 8, loc = pid / 8;
    pid = xcd * qq + (xcd < r ? xcd : r) + loc;
  }
  const int head = pid / ntq, qt = pid % ntq;
  const int64_t hoff = static_cast<int64_t>(head) * ATT_DH;

  // ---- query fragments: block b, lane holds q[row][16 s + 8 hi .. +7] for the 8 k16-steps
  bf16x8 qf[QB][8];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    int qr = qt * C::kQ + (wave * QB + b) * 32 + l32;
    qr = qr < Mq ? qr : Mq - 1;
    const bf16_t* src = q + static_cast<int64_t>(qr) * ldq + hoff + 8 * hi;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[b][s] = __builtin_bit_cast(bf16x8, ldg16(src + 16 * s));
  }

  // ---- direct-load plan: instruction n of this wave fills tile rows 4m .. 4m+3
  // (m = wave + WAVES n); the lane lands in row 4m + lane/16, slot lane%16.
  int k_src[NLD], v_src[NLD], ld_row[NLD], k_off[NLD], v_off[NLD];
#pragma unroll
  for (int n = 0; n < NLD; ++n) {
    const int r = 4 * (wave + WAVES * n) + g16;
    const int p = i16;
    const int ck = k_slot(r, p);                      // the XOR is its own inverse
    const int cv = 2 * v_block(r, p >> 1) + (p & 1);
    ld_row[n] = r;
    k_src[n] = ck * 8;
    v_src[n] = cv * 8;
    k_off[n] = r * static_cast<int>(ldkv) + ck * 8;   // element offsets within a tile
    v_off[n] = r * static_cast<int>(ldkv) + cv * 8;
  }
  const bf16_t* kh = k + hoff;
  const bf16_t* vh = v + hoff;
  const uint32_t lds0 = lds_offset(smem);
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto issue_tile = [&](int t, int stage) __attribute__((always_inline)) {
    const int key0 = t * ATT_KT;
    const uint32_t kdst = lds0 + stage * ATT_STAGE_BYTES;
    const uint32_t vdst = kdst + ATT_TILE_BYTES;
    if (key0 + ATT_KT <= L) {  // full tile: uniform tile base + per-lane offsets
      const bf16_t* kt = kh + static_cast<int64_t>(key0) * ldkv;
      const bf16_t* vt = vh + static_cast<int64_t>(key0) * ldkv;
#pragma unroll
      for (int n = 0; n < NLD; ++n) {
        const uint32_t m = static_cast<uint32_t>(wave_u + WAVES * n);
        lds_copy16(kt + k_off[n], kdst + m * 1024);
        lds_copy16(vt + v_off[n], vdst + m * 1024);
      }
      return;
    }
#pragma unroll
    for (int n = 0; n < NLD; ++n) {
      const uint32_t m = static_cast<uint32_t>(wave_u + WAVES * n);
      int row = key0 + ld_row[n];
      row = row < L ? row : L - 1;  // ragged last tile: re-read row L-1 (finite, masked later)
      const int64_t rofs = static_cast<int64_t>(row) * ldkv;
      lds_copy16(kh + rofs + k_src[n], kdst + m * 1024);
      lds_copy16(vh + rofs + v_src[n], vdst + m * 1024);
    }
  };

  // ---- precomputed LDS read addresses (byte offsets inside a stage)
  // K fragment of k16-step s: row kb*32 + perm23(l32), chunk 2s + hi
  int k_rd[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int r = perm23(l32);
    k_rd[s] = r * 256 + k_slot(r, 2 * s + hi) * 16;
  }
  // V^T operand for dh block d, 16-key step (kb, a), half t: the lane (as a
  // source of the transpose read) addresses row kb*32 + 16a + 8(g16/2) + 4t +
  // i16/4 at dh d*32 + 16(g16%2) + 4(i16%4); it receives V[4 consecutive keys][its dh].
  int v_rd[4][2];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int rlow = 8 * (g16 >> 1) + 4 * t + (i16 >> 2);  // row within the 16-key step
      const int blk = v_block(rlow, 2 * d + (g16 & 1));
      v_rd[d][t] = ATT_TILE_BYTES + rlow * 256 + blk * 32 + 8 * (i16 & 3);
    }

  f32x16 o[QB][4];
#pragma unroll
  for (int b = 0; b < QB; ++b)
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[b][d][r] = 0.0f;
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    m_run[b] = -INFINITY;
    l_run[b] = 0.0f;
  }

  const f32x16 zero16 = {};
  auto compute_s = [&](auto stage_c, f32x16(&sacc)[2][QB]) __attribute__((always_inline)) {
    constexpr int STAGE = decltype(stage_c)::value;
    const char* ks = smem + STAGE * ATT_STAGE_BYTES;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(ks + kb * 32 * 256 + k_rd[s]);
#pragma unroll
        for (int b = 0; b < QB; ++b)
          sacc[kb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              a, qf[b][s], s == 0 ? zero16 : sacc[kb][b], 0, 0, 0);
      }
  };

  auto softmax = [&](f32x16(&sacc)[2][QB], int key0, bf16x8(&pf)[QB][2][2]) __attribute__((always_inline)) {
    if (key0 + ATT_KT > L) {  // ragged last tile: keys past L get -inf
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool valid = key0 + kb * 32 + 16 * (r >> 3) + 8 * hi + (r & 7) < L;
#pragma unroll
          for (int b = 0; b < QB; ++b) sacc[kb][b][r] = valid ? sacc[kb][b][r] : -INFINITY;
        }
    }
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][b][r]);
      mx = pair_max(mx);
      const bool grow = (mx - m_run[b]) * scale_log2 > ATT_RESCALE_LOG2;
      if (__builtin_expect(__ballot(grow) != 0ull, 0)) {
        const float m_new = grow ? mx : m_run[b];
        const float alpha = grow ? __builtin_amdgcn_exp2f((m_run[b] - m_new) * scale_log2) : 1.0f;
        m_run[b] = m_new;
        l_run[b] *= alpha;
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[b][d][r] *= alpha;
      }
      const float neg_mc = -m_run[b] * scale_log2;
      // the row sum adds the bf16 probabilities the PV product uses, two per
      // v_dot2 (fp32 accumulation)
      const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
      float psum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            pf[b][kb][a][j] = static_cast<__bf16>(
                __builtin_amdgcn_exp2f(fmaf(sacc[kb][b][8 * a + j], scale_log2, neg_mc)));
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bf16x2 pair = {pf[b][kb][a][2 * j], pf[b][kb][a][2 * j + 1]};
            psum = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, psum, false);
          }
        }
      l_run[b] += psum;
    }
  };

  auto pv = [&](auto stage_c, const bf16x8(&pf)[QB][2][2]) __attribute__((always_inline)) {
    constexpr int STAGE = decltype(stage_c)::value;
    const char* vs = smem + STAGE * ATT_STAGE_BYTES;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
          const int step = (kb * 32 + 16 * a) * 256;
          const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(ECHO_LDS_V4(vs + step + v_rd[d][0]));
          const v4i16 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16(ECHO_LDS_V4(vs + step + v_rd[d][1]));
          const bf16x8 va = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int b = 0; b < QB; ++b)
            o[b][d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pf[b][kb][a], o[b][d], 0, 0, 0);
        }
  };

  auto softmax_pv = [&](auto stage_c, f32x16(&sacc)[2][QB], int key0) __attribute__((always_inline)) {
    bf16x8 pf[QB][2][2];
    softmax(sacc, key0, pf);
    pv(stage_c, pf);
  };

  const int nkt = (L + ATT_KT - 1) / ATT_KT;
  issue_tile(0, 0);
  if (nkt > 1) issue_tile(1, 1);

  if constexpr (MODE == 1) {
    f32x16 sa[2][QB], sb[2][QB];
    // prologue: tiles 0 and 1 in flight, S(0) computed
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    compute_s(std::integral_constant<int, 0>{}, sa);
    // iteration t: S(t) is in `cur`, tile t sits in stage t%3 and tile t+1 is
    // being loaded into stage (t+1)%3
    auto iteration = [&](auto stage_c, int t, f32x16(&cur)[2][QB], f32x16(&nxt)[2][QB]) __attribute__((always_inline)) {
      constexpr int ST = decltype(stage_c)::value;
      constexpr int ST1 = (ST + 1) % ATT_NSTAGE, ST2 = (ST + 2) % ATT_NSTAGE;
      __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of tile t+1 have landed
      __syncthreads();                // ... everyone's; and stage (t+2)%3 is no longer read
      if (t + 2 < nkt) issue_tile(t + 2, ST2);
      if (t + 1 < nkt) compute_s(std::integral_constant<int, ST1>{}, nxt);
      softmax_pv(std::integral_constant<int, ST>{}, cur, t * ATT_KT);
    };
    // stages cycle with period 3 and the S buffers with period 2: unroll by 6
    for (int t = 0; t < nkt; t += 6) {
      iteration(std::integral_constant<int, 0>{}, t, sa, sb);
      if (t + 1 >= nkt) break;
      iteration(std::integral_constant<int, 1>{}, t + 1, sb, sa);
      if (t + 2 >= nkt) break;
      iteration(std::integral_constant<int, 2>{}, t + 2, sa, sb);
      if (t + 3 >= nkt) break;
      iteration(std::integral_constant<int, 0>{}, t + 3, sb, sa);
      if (t + 4 >= nkt) break;
      iteration(std::integral_constant<int, 1>{}, t + 4, sa, sb);
      if (t + 5 >= nkt) break;
      iteration(std::integral_constant<int, 2>{}, t + 5, sb, sa);
    }
  } else if constexpr (MODE == 0) {
    // iteration t: tile t sits in stage t%3, tile t+1 is in flight
    f32x16 sacc[2][QB];
    auto iteration = [&](auto stage_c, int t) __attribute__((always_inline)) {
      constexpr int ST = decltype(stage_c)::value;
      constexpr int ST2 = (ST + 2) % ATT_NSTAGE;
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(NLD * 2));  // this wave's loads of tile t have landed
      __syncthreads();
      if (t + 2 < nkt) issue_tile(t + 2, ST2);
      compute_s(std::integral_constant<int, ST>{}, sacc);
      softmax_pv(std::integral_constant<int, ST>{}, sacc, t * ATT_KT);
    };
    for (int t = 0; t < nkt; t += 3) {
      iteration(std::integral_constant<int, 0>{}, t);
      if (t + 1 >= nkt) break;
      iteration(std::integral_constant<int, 1>{}, t + 1);
      if (t + 2 >= nkt) break;
      iteration(std::integral_constant<int, 2>{}, t + 2);
    }
  } else {
    // Ping-pong.  Group 1 (the upper half of the waves) runs one phase behind
    // group 0.  Tile t lives in stage t%4: it is read by S(t) in phase A(t)
    // and by PV(t) in phase A(t+1) of both groups, and is overwritten by tile
    // t+4, issued in phase A(t+2).  Before every barrier a wave waits until
    // at most its newest tile's loads are in flight; every wave issues at most
    // one tile between two barriers, so every older tile is complete.  Both
    // groups execute the same number of barriers: group 1 one extra at the
    // start, group 0 one extra at the end.
    const bool late = wave >= WAVES / 2;
    f32x16 sacc[2][QB];
    bf16x8 pf[QB][2][2];
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(NLD * 2));
    __syncthreads();
    if (late) {
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(NLD * 2));
      __syncthreads();
    }
    auto round = [&](auto stage_c, int t) __attribute__((always_inline)) {
      constexpr int ST = decltype(stage_c)::value;           // stage of tile t
      constexpr int STP = (ST + 3) % 4, ST2 = (ST + 2) % 4;  // tiles t-1 and t+2
      // phase A: matrix pipe
      if (t + 2 < nkt) issue_tile(t + 2, ST2);
      if (t > 0) pv(std::integral_constant<int, STP>{}, pf);
      compute_s(std::integral_constant<int, ST>{}, sacc);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(NLD * 2));
      __syncthreads();
      // phase B: vector pipe
      softmax(sacc, t * ATT_KT, pf);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(NLD * 2));
      __syncthreads();
    };
    int t = 0;
    for (; t + 4 <= nkt; t += 4) {
      round(std::integral_constant<int, 0>{}, t);
      round(std::integral_constant<int, 1>{}, t + 1);
      round(std::integral_constant<int, 2>{}, t + 2);
      round(std::integral_constant<int, 3>{}, t + 3);
    }
    // tail rounds (nkt % 4 of them) and the last PV
    const int rem = nkt - t;
    if (rem > 0) round(std::integral_constant<int, 0>{}, t);
    if (rem > 1) round(std::integral_constant<int, 1>{}, t + 1);
    if (rem > 2) round(std::integral_constant<int, 2>{}, t + 2);
    switch ((nkt - 1) & 3) {  // stage of the last tile
      case 0: pv(std::integral_constant<int, 0>{}, pf); break;
      case 1: pv(std::integral_constant<int, 1>{}, pf); break;
      case 2: pv(std::integral_constant<int, 2>{}, pf); break;
      default: pv(std::integral_constant<int, 3>{}, pf); break;
    }
    if (!late) __syncthreads();
  }

  // normalise and write through LDS so that global stores are full 16-byte rows
  __syncthreads();
  bf16_t* Os = reinterpret_cast<bf16_t*>(smem);  // [kQ][ATT_OS_STRIDE]
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const float inv = 1.0f / pair_sum(l_run[b]);
    const int qrow = (wave * QB + b) * 32 + l32;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int dh = d * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
        Os[qrow * ATT_OS_STRIDE + dh] = f32_to_bf16(o[b][d][r] * inv);
      }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < (C::kQ * ATT_DH / 8) / C::kThreads; ++i) {
    const int id = tid + C::kThreads * i;
    const int row = id >> 4, ch = id & 15;
    const int qr = qt * C::kQ + row;
    if (qr < Mq)
      stg16(out + static_cast<int64_t>(qr) * ldo + hoff + ch * 8,
            *reinterpret_cast<const uint4*>(Os + row * ATT_OS_STRIDE + ch * 8));
  }
}

template <int QB, int WAVES, int MODE>
hipError_t launch_attn_variant(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                               int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                               hipStream_t stream) {
  if (Mq <= 0) return hipSuccess;
  typedef AttCfg<QB, WAVES, MODE> C;
  const float scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(ATT_DH)));
  const int ntq = (Mq + C::kQ - 1) / C::kQ;
  return ECHO_LAUNCH("attn_fwd_bf16", (attn_fwd_bf16<QB, WAVES, MODE>), dim3(ntq * H), dim3(C::kThreads), 0,
                     stream, q, ldq, k, v, ldkv, Mq, L, H, scale_log2, out, ldo);
}

hipError_t launch_attn_bf16(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                            int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                            hipStream_t stream) {
  return launch_attn_variant<1, 8, 0>(q, ldq, k, v, ldkv, Mq, L, H, out, ldo, stream);
}

}  // namespace echo

// Restricted-query attention (Sec. 3.3, "Fine-grained latent-level caching"):
// the queries of the selected tokens attend over the keys and values of ALL
// tokens, per head, o = softmax(q k^T / sqrt(dh)) v, dh = 128, bf16 operands
// with fp32 accumulation and an online (streaming) softmax.
//
// gfx950 mapping.  A workgroup of WAVES waves owns WAVES * QB * 32 queries of
// one head (each wave QB blocks of 32 queries).  The build uses 12 waves of
// 32 queries: three waves per SIMD (168 registers each), and each K/V tile
// copied to LDS serves 384 queries (a third fewer copies and barriers per
// query than 8 waves).  Keys stream in tiles of 64:
//   * K and V tiles are copied HBM/L2 -> LDS by direct global-to-LDS loads
//     (global_load_lds_dwordx4: no VGPR staging), row-major [key][dh], into a
//     4-stage ring.  Each lane fetches the 16-byte piece whose swizzled LDS
//     slot is its own lane slot, so the XOR swizzles cost nothing at load time.
//   * S^T (keys x queries) = K_tile . Q^T with v_mfma_f32_32x32x16_bf16; the
//     query fragments stay in registers for the whole key loop; K rows enter
//     the MFMA in a permuted order (bits 2 and 3 of the row index swapped) so
//     that each lane's accumulators hold 8 consecutive keys per 16-key step.
//   * K and V^T fragments flow through a small register ring, each read
//     issued a fixed number of MFMAs ahead of its use.
//   * softmax per lane: a lane owns one query per block (its accumulator
//     column) and half of the tile's keys.  The exp2 argument s c - m c (c =
//     scale log2 e) is one FMA against a per-row reference m c, which is
//     the first half's row maximum and moves only when a half's largest
//     argument exceeds 8 (lazy rescale, by that argument).  No per-tile row
//     maximum is taken: a probability above 2^8 implies a lane sum above
//     2^8, so the common case costs one compare on the row sum; the wave
//     enters the exact path (row maxima, shift, recomputed probabilities)
//     only then, and rows that do not grow get a zero shift and the same
//     values, so each row's arithmetic depends on its own scores only.
//     Masking runs only on the ragged last tile.
//   * O^T (dh x queries) += V^T . P^T: P^T is the S accumulator converted to
//     bf16 in registers; V^T fragments come straight from the row-major V tile
//     with ds_read_b64_tr_b16 (LDS transpose reads), two per 8-key operand.
//   * The key loop is software-pipelined by one half (32 keys): the exp /
//     pack / row sum of half h run between the S MFMAs of half h + 1, and
//     the exp2 arguments of half h + 1 with its first chunks between the PV
//     MFMAs of half h, so that neither phase has much more vector work than
//     matrix work (two accumulator sets for S).
//   * In the steady state a wave's copies of a new tile are issued one at a
//     time between the S MFMAs after the tile barrier, not all at once at the
//     barrier: eight waves issuing their copies together made each wait at
//     the issue of the next copy instead of running its MFMAs (2.7% faster).
// Work balance.  A workgroup holds one CU (its LDS), so (head, query tile)
// items run in rounds of one per CU.  The whole rounds of full items run as
// they are, remapped so that each XCD works through a contiguous range of
// items (the query tiles of one head share that head's K/V stream in one
// L2).  What is left, the leftover full items and the partly filled last
// tile of every head, whose waves without queries skip their matrix work, is
// cut along the keys into ranges of equal cost, and attn_combine merges the
// pieces: the last round ends together instead of taking a whole item's time
// for part of the CUs (32760-token block: 7.27 -> 7.11 ms per call).
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int ATT_KT = 64, ATT_DH = 128;
constexpr int ATT_TILE_BYTES = ATT_KT * ATT_DH * 2;  // one K or V tile: 16 KB
constexpr int ATT_NSTAGE = 4;                         // K/V ring stages
// LDS: the K tiles of the 4 stages, then the V tiles of the 4 stages, so
// that every fragment read is a base register plus a 16-bit immediate offset
constexpr int ATT_V_BASE = ATT_NSTAGE * ATT_TILE_BYTES;  // 64 KB
constexpr int ATT_OS_STRIDE = ATT_DH + 8;            // output staging row (bf16)
constexpr float ATT_RESCALE_LOG2 = 8.0f;             // lazy-rescale headroom (log2 units)
constexpr float ATT_RESCALE_SUM = 256.0f;            // 2^ATT_RESCALE_LOG2
constexpr int ATT_NPRE = 3;     // chunks of a half's softmax done under the PV MFMAs before it
constexpr int ATT_PV_EXP0 = 2;  // PV MFMA after which the first of those chunks takes its exp2
constexpr int ATT_RING = 2;                          // LDS fragment reads in flight per wave

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Four K/V stages: tile t + 3 is copied while S(t+1) and PV(t) run.
template <int QB, int WAVES>
struct AttCfg {
  static constexpr int kThreads = WAVES * 64;
  static constexpr int kQ = WAVES * QB * 32;  // queries per workgroup
  // ring, then (when WAVES does not divide 16) 1 KB per wave with no third piece
  static constexpr int kJunk = 16 % WAVES == 0 ? 0 : 1024 * (WAVES - 16 % WAVES);
  static constexpr int kRingBytes = 2 * ATT_V_BASE + kJunk;
  static constexpr int kLdsBytes = (kRingBytes > kQ * ATT_OS_STRIDE * 2)
                                       ? kRingBytes
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

// one of two register sets, chosen at compile time
template <int I, typename T>
__device__ __forceinline__ T& pick2(T& a, T& b) {
  if constexpr (I == 0)
    return a;
  else
    return b;
}

__device__ __forceinline__ float pair_max(float x) {
  // max over lanes l and l^32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---- work lists.  Items are (head, query tile) pairs in "full first"
// order: item i < nf is full tile i % ntqf of head i / ntqf (ntqf = Mq / kQ
// full tiles per head), item i >= nf the last, partly filled tile of head
// i - nf (present when kQ does not divide Mq).  A launch either takes whole
// items [0, gridDim.x) (mode 0), or the items [first, nf + ns) as a list of
// key tiles weighted by cost (a key tile of a full item costs c_full, one of
// the partly filled item c_part: its waves without queries skip their
// matrix work), cut into gridDim.x ranges of equal cost (mode 1).  A range
// covers whole key tiles of one or more consecutive items; each piece of an
// item it covers is a fragment (a range costs no more than the cheapest item,
// so it holds at most two), whose partial result goes to slot 2 * range +
// (item - first item of the range); attn_combine merges the fragments of
// every item in range order.
struct AttWork {
  int mode;    // 0: whole items, 1: balanced fragments
  int first;   // mode 1: first item of the list
  int c_full;  // mode 1: cost of a key tile of a full item
  int c_part;  // mode 1: cost of a key tile of the partly filled item
  int total;   // mode 1: cost of the whole list (total * gridDim.x < 2^31)
};

struct AttList {
  int ntqf, nf, ns, nkt;
  AttWork w;
  __host__ __device__ AttList(int Mq, int H, int L, int kq, const AttWork& work)
      : ntqf(Mq / kq), nf(H * (Mq / kq)), ns(Mq % kq != 0 ? H : 0), nkt((L + 63) / 64), w(work) {}
  __host__ __device__ int items() const { return nf + ns; }
  __host__ __device__ void item(int i, int& head, int& qt) const {
    head = i < nf ? i / ntqf : i - nf;
    qt = i < nf ? i % ntqf : ntqf;
  }
  // cost of the list before item i (first <= i <= nf + ns)
  __host__ __device__ int prefix(int i) const {
    const int a = (i < nf ? i : nf) - w.first, b = i > nf ? i - nf : 0;
    return (a * w.c_full + b * w.c_part) * nkt;
  }
  // the first key tile whose cost starts at or after x: (item i, tile t)
  __host__ __device__ void locate(int x, int& i, int& t) const {
    const int pf = prefix(nf);
    const int c = x < pf ? w.c_full : w.c_part;
    i = x < pf ? w.first + x / (nkt * w.c_full) : nf + (x - pf) / (nkt * w.c_part);
    t = (x - prefix(i) + c - 1) / c;
    if (t >= nkt) {
      ++i;
      t = 0;
    }
  }
  // start of range g of G, and the range holding the key tile whose cost starts at y
  __host__ __device__ int start(int g, int G) const { return g * w.total / G; }
  __host__ __device__ int owner(int y, int G) const { return ((y + 1) * G - 1) / w.total; }
};

#define ECHO_LDS(p) ((__attribute__((address_space(3))) void*)(p))

#define ECHO_LDS_V4(p) ((__attribute__((address_space(3))) v4i16*)(p))

template <int QB, int WAVES>
__global__ void __launch_bounds__(WAVES * 64, 1)
attn_fwd_bf16(const bf16_t* __restrict__ q, int64_t ldq, const bf16_t* __restrict__ k,
              const bf16_t* __restrict__ v, int64_t ldkv, int Mq, int L, int H, float scale_log2,
              bf16_t* __restrict__ out, int64_t ldo, AttWork work, float* __restrict__ part_o,
              float* __restrict__ part_ml) {
  typedef AttCfg<QB, WAVES> C;
  // Direct-load plan: a K (or V) tile is 16 pieces of 1 KB (piece m = tile
  // rows 4m .. 4m+3).  When WAVES divides 16, wave w copies the K and V
  // pieces w + WAVES n.  Otherwise (12 waves) every wave copies three pieces:
  // K piece w, V piece w, and a third one: K piece 12 + w for waves 0-3,
  // V piece 12 + (w - 4) for waves 4-7, and for waves 8-11 a re-copy of one
  // lane's 16 bytes of its K row into a private 1 KB LDS area nobody reads,
  // so that every wave has the same copy count and no branch.
  constexpr bool EVEN = 16 % WAVES == 0;
  constexpr int NLD = EVEN ? 16 / WAVES : 1;  // K (and V) pieces per wave in the regular slots
  constexpr int NC = EVEN ? 2 * NLD : 3;      // copies per wave per tile
  static_assert(EVEN || (WAVES == 12 && 16 - WAVES == 4), "12 waves: 4 extra K and 4 extra V pieces");
  __shared__ __attribute__((aligned(1024))) char smem[C::kLdsBytes];


  // Mode 0: item blockIdx.x, remapped so that each XCD works through a
  // contiguous range of items, all its key tiles, output written here.
  // Mode 1: the fragments of range blockIdx.x of the weighted list, partial
  // results for attn_combine.
  const AttList list(Mq, H, L, C::kQ, work);
  const int nkt_all = list.nkt;
  const bool split = work.mode == 1;
  int i_s, t_s, i_e, t_e;  // first key tile of the range, first key tile past it
  if (!split) {
    const int total = gridDim.x;
    const int pid = blockIdx.x;
    const int qq = total / 8, r = total % 8, xcd = pid % 8, loc = pid / 8;
    i_s = i_e = xcd * qq + (xcd < r ? xcd : r) + loc;
    t_s = 0;
    t_e = nkt_all;
  } else {
    list.locate(list.start(blockIdx.x, gridDim.x), i_s, t_s);
    list.locate(list.start(blockIdx.x + 1, gridDim.x), i_e, t_e);
  }
  // A range holds at most two fragments (it costs no more than the cheapest
  // item): the tail of one item, the head of the next.  Unrolled, so that
  // the second runs as straight-line code after the first.
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int item = i_s + f;
    if (!(item < i_e || (item == i_e && (f == 0 ? t_s : 0) < t_e))) break;  // uniform per workgroup
    // every wave is done with the stages (and the output staging) of the
    // fragment before
    if (f == 1) __syncthreads();
    // the thread index through an empty asm, so that the compiler computes
    // every lane-dependent address of the fragment here, not once ahead of the
    // fragment loop with its registers held through every key loop
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int wave = tid / kWave, lane = tid % kWave, l32 = lane & 31, hi = lane >> 5;
    const int g16 = lane >> 4, i16 = lane & 15;
    int head, qt;
    list.item(item, head, qt);
    const int t_begin = f == 0 ? t_s : 0;                           // first key tile of the fragment
    const int nkt = (item == i_e ? t_e : nkt_all) - t_begin;        // >= 1
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
    // The query loads are the only memory reads the compiler tracks (the tile
    // copies are inline assembly): waiting for them here keeps it from placing
    // vmcnt waits before their first use inside the loop, where the hardware
    // counter also holds the copies of the next two tiles.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

    // ---- direct-load plan: regular slot n of this wave holds K and V piece
    // m = wave + WAVES n; the lane lands in row 4m + lane/16, slot lane%16.
    // Bits 0-3 of the row, and with them the swizzled slots, are the same for
    // every piece of a wave (WAVES is a multiple of 4).
    static_assert(WAVES % 4 == 0, "row bits 0-3 shared by a wave's pieces");
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const uint32_t ldkv2 = static_cast<uint32_t>(ldkv) * 2u;
    uint32_t row_off[NLD];  // byte offset of the lane's row within a tile
#pragma unroll
    for (int n = 0; n < NLD; ++n) row_off[n] = static_cast<uint32_t>(4 * (wave_u + WAVES * n) + g16) * ldkv2;
    const int r0 = 4 * wave_u + g16;
    const uint32_t k_src = static_cast<uint32_t>(k_slot(r0, i16) * 16);  // the XOR is its own inverse
    const uint32_t v_src = static_cast<uint32_t>((2 * v_block(r0, i16 >> 1) + (i16 & 1)) * 16);
    // third piece (uneven plans): K piece 12 + w (w < 4), V piece 8 + w
    // (4 <= w < 8), else the private area; x_off is the piece's destination
    // within a stage, or the area's absolute LDS offset
    const bool x_v = !EVEN && wave_u >= 4 && wave_u < 8;
    const bool x_junk = !EVEN && wave_u >= 8;
    const int x_piece = wave_u < 4 ? 12 + wave_u : 8 + wave_u;
    const uint32_t x_row = x_junk ? row_off[0] : static_cast<uint32_t>(4 * x_piece + g16) * ldkv2;
    const uint32_t x_src = x_v ? v_src : k_src;
    const uint32_t lds0 = lds_offset(smem);
    const uint32_t x_off = x_junk ? lds0 + 2 * ATT_V_BASE + (wave_u - 8) * 1024
                                  : (x_v ? ATT_V_BASE : 0) + x_piece * 1024;
    const bf16_t* kh = k + hoff;
    const bf16_t* vh = v + hoff;
    // the re-copies of waves 8-11 run on one lane (16 bytes into the private
    // area instead of 1 KB; each still counts once in vmcnt): attention 7.451
    // -> 7.435 ms per call on the 32760-token block
    const uint64_t x_exec = x_junk ? 1ull : ~0ull;

    // Copies of relative tile t into a stage, issued one at a time:
    // tile_prep() takes the tile's sources and stage; tile_copy(c) issues copy
    // c (K then V of regular piece c / 2; the third piece last).  Branch-free:
    // the tile start is part of the uniform base and each lane clamps its row
    // offset to the row L - 1 (rows past L are finite copies of row L - 1,
    // masked later); a tile index past the last tile re-copies the last tile
    // (into a stage that is free), so every wave always has the copies of
    // exactly two tiles in flight after an issue and one wait count fits every
    // iteration.
    const bf16_t* pk_src = kh;
    const bf16_t* pv_src = vh;
    uint32_t p_last = 0, p_kdst = 0;
    auto tile_prep = [&](int t, int stage) __attribute__((always_inline)) {
      t = t < nkt ? t : nkt - 1;
      const int key0 = (t_begin + t) * ATT_KT;
      pk_src = kh + static_cast<int64_t>(key0) * ldkv;
      pv_src = vh + static_cast<int64_t>(key0) * ldkv;
      p_last = static_cast<uint32_t>(L - 1 - key0) * ldkv2;  // offset of row L - 1
      p_kdst = lds0 + stage * ATT_TILE_BYTES;
    };
    auto tile_copy = [&](int c) __attribute__((always_inline)) {
      if (!EVEN && c == 2) {
        const uint32_t ro = x_row < p_last ? x_row : p_last;
        lds_copy16_s_exec(x_v ? pv_src : pk_src, ro + x_src, x_junk ? x_off : p_kdst + x_off, x_exec);
        return;
      }
      const int n = c / 2;
      const uint32_t m = static_cast<uint32_t>(wave_u + WAVES * n);
      const uint32_t ro = row_off[n] < p_last ? row_off[n] : p_last;
      if (c % 2 == 0)
        lds_copy16_s(pk_src, ro + k_src, p_kdst + m * 1024);
      else
        lds_copy16_s(pv_src, ro + v_src, p_kdst + ATT_V_BASE + m * 1024);
    };
    auto issue_tile = [&](int t, int stage) __attribute__((always_inline)) {
      tile_prep(t, stage);
#pragma unroll
      for (int c = 0; c < NC; ++c) tile_copy(c);
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
    // (half t adds 4 rows: the swizzle depends on row bits 0-1 only, so the
    // second address is the first + 1024, an immediate offset)
    int v_rd[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int rlow = 8 * (g16 >> 1) + (i16 >> 2);  // row within the 16-key step (half 0)
      const int blk = v_block(rlow, 2 * d + (g16 & 1));
      v_rd[d] = ATT_V_BASE + rlow * 256 + blk * 32 + 8 * (i16 & 3);
    }

    f32x16 o[QB][4];
#pragma unroll
    for (int b = 0; b < QB; ++b)
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[b][d][r] = 0.0f;
    // mc: the row's reference maximum times scale_log2 (exp2 units); l_run:
    // running sum of the probabilities, relative to the same reference
    float mc[QB], l_run[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) l_run[b] = 0.0f;

    const f32x16 zero16 = {};
    const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};

    // The key loop works in halves of 32 keys: half h is key block kb = h % 2
    // of tile h / 2.  A lane holds 16 scores of a half per query block (its
    // accumulator column; lanes l and l ^ 32 share a query).
    //
    // K fragment of S step st (k16 block of dh) for key block kb of a stage
    auto read_k = [&](const char* ks, int kb, int st) __attribute__((always_inline)) {
      return *reinterpret_cast<const bf16x8*>(ks + kb * 32 * 256 + k_rd[st]);
    };
    // V^T fragment of PV step (d, a) for key block kb: dh block d, 16-key half a
    auto read_v = [&](const char* vs, int kb, int d, int a) __attribute__((always_inline)) {
      const int step = (kb * 32 + 16 * a) * 256;
      const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(ECHO_LDS_V4(vs + step + v_rd[d]));
      const v4i16 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16(ECHO_LDS_V4(vs + step + v_rd[d] + 4 * 256));
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    // Fragments flow through a ring of ATT_RING registers: the read for step
    // i + ATT_RING is issued right after the MFMA of step i has taken its
    // operand, so every MFMA finds its fragment ATT_RING steps old.
    //
    // S of one half (8 MFMAs) with `work(i)` placed after MFMA i
    auto s_half = [&](const char* ks, int kb, f32x16(&sh)[QB], auto&& work) __attribute__((always_inline)) {
      bf16x8 ring[ATT_RING];
#pragma unroll
      for (int i = 0; i < ATT_RING; ++i) ring[i] = read_k(ks, kb, i);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bf16x8 a = ring[i % ATT_RING];
#pragma unroll
        for (int b = 0; b < QB; ++b)
          sh[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[b][i], i == 0 ? zero16 : sh[b], 0, 0, 0);
        if (i + ATT_RING < 8) ring[i % ATT_RING] = read_k(ks, kb, i + ATT_RING);
        work(i);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // O += V^T P^T for one half (8 MFMAs: 16-key half a = i / 4, dh block
    // d = i % 4, so that the first four use only the probabilities of keys
    // 0-15) with `work(i)` placed after MFMA i
    auto pv_half = [&](const char* vs, int kb, const bf16x8(&pf)[QB][2], auto&& work) __attribute__((always_inline)) {
      bf16x8 ring[ATT_RING];
#pragma unroll
      for (int i = 0; i < ATT_RING; ++i) ring[i] = read_v(vs, kb, i % 4, i / 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int d = i % 4, a = i / 4;
        const bf16x8 va = ring[i % ATT_RING];
#pragma unroll
        for (int b = 0; b < QB; ++b)
          o[b][d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pf[b][a], o[b][d], 0, 0, 0);
        if (i + ATT_RING < 8) ring[i % ATT_RING] = read_v(vs, kb, (i + ATT_RING) % 4, (i + ATT_RING) / 4);
        work(i);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // keys past L (ragged last tile) get -inf; keyh = first key of the half
    auto mask_half = [&](f32x16(&sh)[QB], int keyh) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool valid = keyh + 16 * (r >> 3) + 8 * hi + (r & 7) < L;
#pragma unroll
        for (int b = 0; b < QB; ++b) sh[b][r] = valid ? sh[b][r] : -INFINITY;
      }
    };
    // Softmax of a half in chunks of two scores (chunk c: elements 2c, 2c + 1,
    // probabilities pf[b][c / 4][2 (c % 4) ..]).  Three steps, placed apart:
    // the exp2 argument s scale_log2 - mc, in place; its exp2; the bf16 pack
    // (the PV operand) and the row sum of the same bf16 values, two per v_dot2.
    auto arg_chunk = [&](f32x16(&sh)[QB], int c) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        sh[b][2 * c] = fmaf(sh[b][2 * c], scale_log2, -mc[b]);
        sh[b][2 * c + 1] = fmaf(sh[b][2 * c + 1], scale_log2, -mc[b]);
      }
    };
    auto exp_chunk = [&](const f32x16(&sh)[QB], int c, float(&t)[QB][2]) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        t[b][0] = __builtin_amdgcn_exp2f(sh[b][2 * c]);
        t[b][1] = __builtin_amdgcn_exp2f(sh[b][2 * c + 1]);
      }
    };
    bf16x8 pf[QB][2];
    float psum[QB];
    auto pack_chunk = [&](int c, const float(&t)[QB][2]) __attribute__((always_inline)) {
      const int a = c / 4, j = 2 * (c % 4);
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        pf[b][a][j] = static_cast<__bf16>(t[b][0]);
        pf[b][a][j + 1] = static_cast<__bf16>(t[b][1]);
        const bf16x2 pair = {pf[b][a][j], pf[b][a][j + 1]};
        psum[b] = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, psum[b], false);
      }
    };
    // Lazy rescale.  The arguments are taken against the reference mc; a row
    // moves its reference only when the half's largest argument exceeds
    // ATT_RESCALE_LOG2 (its maximum grew by more than 2^8), by that argument.
    // No probability can exceed 2^8 unless the lane's sum does, so the common
    // case costs one compare on the sum; the wave enters the exact path only
    // when some lane's sum is above 2^8.  There, rows that do not grow get a
    // shift of 0 and recompute the same values: each row's arithmetic depends
    // on its own scores only.
    auto settle_exact = [&](f32x16(&sh)[QB]) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        float mx = sh[b][0];
#pragma unroll
        for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sh[b][r]);
        mx = pair_max(mx);
        const float d = mx > ATT_RESCALE_LOG2 ? mx : 0.0f;
        const float alpha = __builtin_amdgcn_exp2f(-d);
        mc[b] += d;
        l_run[b] *= alpha;
#pragma unroll
        for (int dd = 0; dd < 4; ++dd)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[b][dd][r] *= alpha;
#pragma unroll
        for (int r = 0; r < 16; ++r) sh[b][r] -= d;
        psum[b] = 0.0f;
      }
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        float t[QB][2];
        exp_chunk(sh, c, t);
        pack_chunk(c, t);
      }
    };
    auto any_big = [&]() __attribute__((always_inline)) {
      bool big = false;
#pragma unroll
      for (int b = 0; b < QB; ++b) big = big || psum[b] > ATT_RESCALE_SUM;
      return __ballot(big) != 0ull;
    };
    auto add_sum = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < QB; ++b) l_run[b] += psum[b];
    };
    // A half's softmax starts (arguments of all chunks, probabilities of chunks
    // 0 .. ATT_NPRE - 1) under the PV MFMAs of the half before it and finishes
    // under the S MFMAs of the half after it.
    constexpr int NPRE = ATT_NPRE, NJ = 8 - NPRE;
    auto begin_half = [&](f32x16(&sh)[QB]) __attribute__((always_inline)) {
#pragma unroll
      for (int c = 0; c < 8; ++c) arg_chunk(sh, c);
#pragma unroll
      for (int b = 0; b < QB; ++b) psum[b] = 0.0f;
#pragma unroll
      for (int c = 0; c < NPRE; ++c) {
        float t[QB][2];
        exp_chunk(sh, c, t);
        pack_chunk(c, t);
      }
    };
    auto finish_half = [&](f32x16(&sh)[QB]) __attribute__((always_inline)) {
#pragma unroll
      for (int c = NPRE; c < 8; ++c) {
        float t[QB][2];
        exp_chunk(sh, c, t);
        pack_chunk(c, t);
      }
      if (__builtin_expect(any_big(), 0)) settle_exact(sh);
      add_sum();
    };

    // ---- the key loop, software-pipelined by one half.  Half h starts with
    // the arguments of S_h in one accumulator set and its first NPRE chunks
    // packed:
    //   at a tile boundary (h + 1 even): wait for tile (h + 1) / 2; barrier
    //     (every wave is past the PV of tile (h + 1) / 2 - 2, whose stage is
    //     free); issue tile (h + 1) / 2 + 2;
    //   A: the 8 MFMAs of S_{h+1}  +  exp / pack / row sum of the rest of half h;
    //      settle half h (lazy rescale, row sum);
    //   B: the 8 MFMAs of PV_h     +  arguments of S_{h+1}, its first chunks.
    // Each wave's vector work thus runs under its own matrix work.  The
    // steady state runs in blocks of 8 halves (4 tiles, one turn of the stage
    // ring) whose halves have no key past L, as straight-line code; the
    // remaining halves, the ragged one included, take a plain per-half path.
    // Tiles are counted from t_begin.
    const int key_begin = t_begin * ATT_KT;
    const int nh = 2 * nkt;
    const int nh_full = (L - key_begin) / 32 < nh ? (L - key_begin) / 32 : nh;  // halves with no key past L
    auto boundary = [&](int t, int stage_next2) __attribute__((always_inline)) {
      // this wave's copies of tile t have landed; those of tile t + 1 may be in flight
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(NC));
      __syncthreads();
      issue_tile(t + 2, stage_next2);
    };
    // A wave whose query blocks all lie past Mq (waves of the last, partly
    // filled query tile of a head) skips the matrix and softmax work: it
    // issues its share of the tile copies and meets the others at the same
    // nkt barriers.
    const bool idle = qt * C::kQ + wave * QB * 32 >= Mq;  // uniform per wave
    f32x16 s0[QB], s1[QB];
    issue_tile(0, 0);
    issue_tile(1, 1);
    if (idle) {
      for (int t = 0; t < nkt; ++t) boundary(t, (t + 2) % ATT_NSTAGE);
    } else {
      boundary(0, 2);
      {
        s_half(smem, 0, s0, [](int) {});
        if (key_begin + 32 > L) mask_half(s0, key_begin);
        // the first reference: the row maximum of the first half (every row has
        // a key there)
#pragma unroll
        for (int b = 0; b < QB; ++b) {
          float mx = s0[b][0];
#pragma unroll
          for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s0[b][r]);
          mc[b] = pair_max(mx) * scale_log2;
        }
        begin_half(s0);
      }

      // H = h % 8: tile h / 2 in stage H / 2, key block H % 2, S_h in set H % 2
      auto half_step = [&](auto h_c, int h) __attribute__((always_inline)) {
        constexpr int H = decltype(h_c)::value;
        constexpr int ST = H / 2, KB = H % 2;
        constexpr int HN = (H + 1) % 8, STN = HN / 2, KBN = HN % 2;
        auto& sc = pick2<KB>(s0, s1);
        auto& sn = pick2<1 - KB>(s0, s1);
        if constexpr (KBN == 0) {
          // this wave's copies of the new tile have landed; after the barrier
          // every wave is past the tile whose stage the copies below refill
          __builtin_amdgcn_s_waitcnt(waitcnt_vm(NC));
          __syncthreads();
          tile_prep((h + 1) / 2 + 2, (STN + 2) % ATT_NSTAGE);
        }
        // chunk NPRE + j: exp2 after S MFMA 8 j / NJ, pack and row sum after the next
        float tq[2][QB][2];
        // the wave's S phase (with the exp work of the half before) at a higher
        // issue priority than the PV phases of the other waves on its SIMD
        // (0.5% faster; the reverse was 1.3% slower)
        __builtin_amdgcn_s_setprio(2);
        s_half(smem + STN * ATT_TILE_BYTES, KBN, sn, [&](int i) __attribute__((always_inline)) {
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            if (i == (8 * j) / NJ) exp_chunk(sc, NPRE + j, tq[j % 2]);
            if (i == (8 * j) / NJ + 1) pack_chunk(NPRE + j, tq[j % 2]);
          }
          if constexpr (KBN == 0) {
            // the wave's NC copies of the tile, spread evenly over the 8 MFMAs
#pragma unroll
            for (int c = (i * NC) / 8; c < ((i + 1) * NC) / 8; ++c) tile_copy(c);
          }
        });
        // the arguments of S_h are gone (their registers were reused as the
        // chunks finished); the exact path recomputes S_h from the K tile, still
        // in its stage, by the same MFMA sequence (the same values)
        if (__builtin_expect(any_big(), 0)) {
          f32x16 sr[QB];
          s_half(smem + ST * ATT_TILE_BYTES, KB, sr, [](int) {});
#pragma unroll
          for (int c = 0; c < 8; ++c) arg_chunk(sr, c);
          settle_exact(sr);
        }
        add_sum();
#pragma unroll
        for (int b = 0; b < QB; ++b) psum[b] = 0.0f;
        // S_{h+1}: arguments of chunks 0 .. NPRE - 1 after PV MFMA 0, their exp2
        // after MFMAs 2 .., each pack one MFMA later (the first four PV MFMAs read
        // the packed keys 0-15); the other arguments after MFMAs 4-7
        __builtin_amdgcn_s_setprio(0);
        pv_half(smem + ST * ATT_TILE_BYTES, KB, pf, [&](int i) __attribute__((always_inline)) {
          if (i == 0) {
#pragma unroll
            for (int c = 0; c < NPRE; ++c) arg_chunk(sn, c);
          }
#pragma unroll
          for (int c = 0; c < NPRE; ++c) {
            if (i == ATT_PV_EXP0 + c) exp_chunk(sn, c, tq[c % 2]);
            if (i == ATT_PV_EXP0 + 1 + c) pack_chunk(c, tq[c % 2]);
          }
#pragma unroll
          for (int k = 0; k < NJ; ++k)
            if (i == 4 + (4 * k) / NJ) arg_chunk(sn, NPRE + k);
        });
      };
      int h = 0;
      for (; h + 8 < nh_full; h += 8) {
        half_step(std::integral_constant<int, 0>{}, h);
        half_step(std::integral_constant<int, 1>{}, h + 1);
        half_step(std::integral_constant<int, 2>{}, h + 2);
        half_step(std::integral_constant<int, 3>{}, h + 3);
        half_step(std::integral_constant<int, 4>{}, h + 4);
        half_step(std::integral_constant<int, 5>{}, h + 5);
        half_step(std::integral_constant<int, 6>{}, h + 6);
        half_step(std::integral_constant<int, 7>{}, h + 7);
      }
      // The remaining halves one at a time (S_h is in s0, tile h / 2 in stage 0).
      for (; h < nh; ++h) {
        finish_half(s0);
        pv_half(smem + ((h / 2) % ATT_NSTAGE) * ATT_TILE_BYTES, h % 2, pf, [](int) {});
        if (h + 1 < nh) {
          const int hn = h + 1, stn = (hn / 2) % ATT_NSTAGE;
          if (hn % 2 == 0) boundary(hn / 2, (stn + 2) % ATT_NSTAGE);
          s_half(smem + stn * ATT_TILE_BYTES, hn % 2, s0, [](int) {});
          const int keyh = key_begin + hn * 32;
          if (keyh + 32 > L) mask_half(s0, keyh);
          begin_half(s0);
        }
      }
    }  // !idle
    // drain the copies still in flight (re-copies past the last tile) before
    // the LDS is reused, the next fragment starts or the workgroup ends
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

    if (split) {
      // fragment: unnormalised output in the accumulator layout (for each
      // (b, d, r) the 64 lanes write 256 contiguous bytes), reference maximum
      // (exp2 units) and row sum per query; waves without queries write nothing
      if (idle) continue;
      const int64_t unit = 2 * static_cast<int64_t>(blockIdx.x) + f;
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const float lsum = pair_sum(l_run[b]);
        const int qloc = (wave * QB + b) * 32 + l32;
        if (hi == 0) {
          part_ml[(unit * C::kQ + qloc) * 2] = mc[b];
          part_ml[(unit * C::kQ + qloc) * 2 + 1] = lsum;
        }
        float* po = part_o + ((unit * WAVES + wave) * QB + b) * (4 * 16 * kWave);
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) po[(d * 16 + r) * kWave + lane] = o[b][d][r];
      }
      continue;
    }

    // normalise and write through LDS so that global stores are full 16-byte rows
    __syncthreads();
    bf16_t* Os = reinterpret_cast<bf16_t*>(smem);  // [kQ][ATT_OS_STRIDE]
#pragma unroll
    for (int b = 0; b < QB && !idle; ++b) {
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
  }  // fragments
}

constexpr int ATT_MAX_RANGES = 1024;  // ranges of a balanced list

// Merge the fragments of the items of a balanced list: o = sum_s 2^{r_s - r}
// o_s / sum_s 2^{r_s - r} l_s, where r_s is fragment s's reference maximum in
// exp2 units (times scale log2 e) and r = max_s r_s, fragments added in key
// order.  One workgroup per 32-query block of an item: its threads take the
// block's 4096 outputs in the order the partials are stored (the accumulator
// layout: lane fastest), so every fragment's partial is read with consecutive
// addresses, and the bf16 results go through LDS so that the output is
// written as 16-byte row pieces (2-byte stores scattered over 32 rows wrote
// partial lines: 34.0 -> 25.5 us per call on the 32760-token block).  A
// thread's 16 outputs belong to one query, so it forms that query's fragment
// weights once and reads each fragment's 16 partials together (about 30 us
// less per call on the 32760-token block, bit-identical).
template <int QB, int WAVES>
__global__ void __launch_bounds__(256)
attn_combine(const float* __restrict__ part_o, const float* __restrict__ part_ml, AttWork work, int G,
             int Mq, int L, int H, bf16_t* __restrict__ out, int64_t ldo) {
  typedef AttCfg<QB, WAVES> C;
  constexpr int64_t kUnit = static_cast<int64_t>(C::kQ) * ATT_DH;  // partial floats per unit
  constexpr int kBlk = 32 * ATT_DH;                                // partial floats per 32-query block
  constexpr int kBlocks = C::kQ / 32;                              // 32-query blocks per item
  static_assert(kBlk % 256 == 0, "whole passes of the workgroup");
  __shared__ __attribute__((aligned(16))) bf16_t Os[32 * ATT_OS_STRIDE];
  __shared__ int64_t units[ATT_MAX_RANGES];
  const AttList list(Mq, H, L, C::kQ, work);
  const int item = work.first + static_cast<int>(blockIdx.x) / kBlocks, wb = blockIdx.x % kBlocks;
  if (item >= list.items()) return;  // uniform per workgroup
  int head, qt;
  list.item(item, head, qt);
  const int q0 = qt * C::kQ + wb * 32;  // first query of the block
  if (q0 >= Mq) return;
  // the item's fragments: ranges g0 .. g1, each its slot (item - first item of the range)
  const int p0 = list.prefix(item);
  const int c = item < list.nf ? work.c_full : work.c_part;
  const int g0 = list.owner(p0, G), g1 = list.owner(p0 + (list.nkt - 1) * c, G);
  const int nfrag = g1 - g0 + 1;  // <= G <= ATT_MAX_RANGES
  for (int f = static_cast<int>(threadIdx.x); f < nfrag; f += 256) {
    int i0, t0;
    list.locate(list.start(g0 + f, G), i0, t0);
    units[f] = 2 * static_cast<int64_t>(g0 + f) + (item - i0);
  }
  __syncthreads();
  // thread t takes the block's outputs t + 256 k (storage order (d * 16 + r)
  // * 64 + lane): its lane, hence its query, is the same for every k, so the
  // query's fragment weights are formed once and each fragment's 16 partials
  // are read together
  constexpr int KS = kBlk / 256;
  const int tid = static_cast<int>(threadIdx.x);
  const int l32 = tid % kWave & 31, qloc = wb * 32 + l32;
  float m = -INFINITY;
  for (int f = 0; f < nfrag; ++f) m = fmaxf(m, part_ml[(units[f] * C::kQ + qloc) * 2]);
  float lsum = 0.0f, acc[KS];
#pragma unroll
  for (int k = 0; k < KS; ++k) acc[k] = 0.0f;
  for (int f = 0; f < nfrag; ++f) {
    const int64_t unit = units[f];
    const float w = __builtin_amdgcn_exp2f(part_ml[(unit * C::kQ + qloc) * 2] - m);
    lsum += w * part_ml[(unit * C::kQ + qloc) * 2 + 1];
    const float* po = part_o + unit * kUnit + wb * kBlk + tid;
#pragma unroll
    for (int k = 0; k < KS; ++k) acc[k] += w * po[256 * k];
  }
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const int e = tid + 256 * k;
    const int lane = e % kWave, dr = e / kWave;
    const int d = dr / 16, r = dr % 16, hi = lane >> 5;
    const int dh = d * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
    Os[l32 * ATT_OS_STRIDE + dh] = f32_to_bf16(acc[k] / lsum);
  }
  __syncthreads();
  // the block's 32 rows, 16 pieces of 16 bytes each
  for (int cc = static_cast<int>(threadIdx.x); cc < 32 * (ATT_DH / 8); cc += 256) {
    const int row = cc / (ATT_DH / 8), ch = cc % (ATT_DH / 8);
    const int qg = q0 + row;
    if (qg < Mq)
      stg16(out + static_cast<int64_t>(qg) * ldo + static_cast<int64_t>(head) * ATT_DH + ch * 8,
            *reinterpret_cast<const uint4*>(Os + row * ATT_OS_STRIDE + ch * 8));
  }
}

// Costs of a key tile in the balanced list, in sixteenths of a full item's:
// the partly filled item runs only the waves that hold queries, so its cost
// follows the most waves with queries on one SIMD (1, 2 or 3 of 3; measured
// over 32760 keys, one item per head on 40 CUs: 48, 160 and 288 queries take
// 0.49, 0.68 and 0.97 of the time of 384).
constexpr int ATT_COST_FULL = 16;
constexpr int ATT_COST_PART[3] = {8, 11, 16};
// Below this many key tiles per item the fragments' set-up outweighs what
// the balance saves, and every item runs whole in one launch.
constexpr int ATT_MIN_BALANCE_TILES = 32;

struct AttPlan {
  bool balanced;  // else one launch of whole items
  int A;          // whole rounds of full items run whole, before the list
  int G;          // ranges of the balanced list
  AttWork w;
  size_t bytes;   // partial results of the list
};

// Items [0, A) (whole rounds of full items, one workgroup per CU: the LDS
// allows one) run whole; the rest, the leftover full items and the partly
// filled ones, is cut into k ranges of equal cost per CU, k the least that
// keeps a range within the cost of the cheapest item, so that the last
// round ends together (a range with one piece of each of two items takes
// the same time as any other, whichever CU the workgroup lands on).
template <int KQ>
AttPlan att_plan(int Mq, int L, int H, int ncu) {
  AttPlan p{};
  AttWork w{};
  const AttList shape(Mq, H, L, KQ, w);
  p.A = shape.nf / ncu * ncu;
  const int rest = shape.items() - p.A;
  if (rest == 0 || shape.nkt < ATT_MIN_BALANCE_TILES) return p;
  const int rem = Mq - shape.ntqf * KQ;
  const int per_simd = ((rem + 31) / 32 + 3) / 4;  // waves with queries on the busiest SIMD
  w.mode = 1;
  w.first = p.A;
  w.c_full = ATT_COST_FULL;
  w.c_part = ATT_COST_PART[(per_simd >= 1 ? per_simd : 1) - 1];
  // costs in 32 bits: total * G < 2^31
  const long long total = (static_cast<long long>(shape.nf - p.A) * w.c_full +
                           static_cast<long long>(shape.ns) * w.c_part) * shape.nkt;
  // k * ncu ranges of equal cost, k the least that keeps every range within
  // the cost of the cheapest item (at most two fragments per range): each CU
  // then runs k ranges, whatever the order the workgroups are dealt in
  const long long c_min = static_cast<long long>(w.c_part < w.c_full && shape.ns > 0 ? w.c_part : w.c_full) *
                          shape.nkt;
  const long long kr = (total + c_min * ncu - 1) / (c_min * ncu);
  // and no more ranges than full-item key tiles' worth of cost, so that every
  // range holds at least one key tile
  const long long G = kr * ncu < total / w.c_full ? kr * ncu : total / w.c_full;
  if (kr > 3 || G < 1 || G > ATT_MAX_RANGES || total * G >= (1ll << 31)) return p;
  w.total = static_cast<int>(total);
  // every range holds at most two fragments (by the cost bound; checked)
  const AttList list(Mq, H, L, KQ, w);
  for (int g = 0; g < static_cast<int>(G); ++g) {
    int i_s, t_s, i_e, t_e;
    list.locate(list.start(g, static_cast<int>(G)), i_s, t_s);
    list.locate(list.start(g + 1, static_cast<int>(G)), i_e, t_e);
    const int n = i_e - i_s + ((i_e == i_s ? t_s : 0) < t_e ? 1 : 0);
    if (n < 1 || n > 2) return p;
  }
  p.G = static_cast<int>(G);
  p.w = w;
  p.bytes = sizeof(float) * static_cast<size_t>(p.G) * 2 * KQ * (ATT_DH + 2);
  p.balanced = true;
  return p;
}

template <int QB, int WAVES>
hipError_t launch_attn_variant(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                               int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                               float* part, size_t part_bytes, hipStream_t stream, const char* name) {
  if (Mq <= 0) return hipSuccess;
  typedef AttCfg<QB, WAVES> C;
  const float scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(ATT_DH)));
  const AttPlan plan = att_plan<C::kQ>(Mq, L, H, device_cu_count());
  ::echo::TimedLaunch scope(name, stream);
  AttWork whole{};
  if (!plan.balanced || part == nullptr || part_bytes < plan.bytes) {
    const int items = AttList(Mq, H, L, C::kQ, whole).items();
    hipLaunchKernelGGL((attn_fwd_bf16<QB, WAVES>), dim3(items), dim3(C::kThreads), 0, stream, q, ldq, k, v,
                       ldkv, Mq, L, H, scale_log2, out, ldo, whole, nullptr, nullptr);
    return hipGetLastError();
  }
  if (plan.A > 0) {
    hipLaunchKernelGGL((attn_fwd_bf16<QB, WAVES>), dim3(plan.A), dim3(C::kThreads), 0, stream, q, ldq, k, v,
                       ldkv, Mq, L, H, scale_log2, out, ldo, whole, nullptr, nullptr);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  float* part_o = part;
  float* part_ml = part + static_cast<size_t>(plan.G) * 2 * C::kQ * ATT_DH;
  hipLaunchKernelGGL((attn_fwd_bf16<QB, WAVES>), dim3(plan.G), dim3(C::kThreads), 0, stream, q, ldq, k,
                     v, ldkv, Mq, L, H, scale_log2, out, ldo, plan.w, part_o, part_ml);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rest = AttList(Mq, H, L, C::kQ, whole).items() - plan.A;
  hipLaunchKernelGGL((attn_combine<QB, WAVES>), dim3(static_cast<unsigned>(rest * (C::kQ / 32))), dim3(256), 0,
                     stream, part_o, part_ml, plan.w, plan.G, Mq, L, H, out, ldo);
  return hipGetLastError();
}

size_t attn_partial_bytes(int Mq_max, int L, int H) {
  // a balanced list has at most min(3 CUs' worth, its key tiles) ranges of two pieces
  typedef AttCfg<1, 12> C;
  const long long nkt = (L + ATT_KT - 1) / ATT_KT;
  if (Mq_max <= 0 || nkt < ATT_MIN_BALANCE_TILES) return 0;
  const long long tiles = static_cast<long long>(H) * ((Mq_max + C::kQ - 1) / C::kQ) * nkt;
  long long G = 3ll * device_cu_count();
  G = G < tiles ? G : tiles;
  G = G < ATT_MAX_RANGES ? G : ATT_MAX_RANGES;
  return sizeof(float) * static_cast<size_t>(G) * 2 * C::kQ * (ATT_DH + 2);
}

hipError_t launch_attn_bf16(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                            int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                            float* part, size_t part_bytes, hipStream_t stream, const char* timing_name) {
  return launch_attn_variant<1, 12>(q, ldq, k, v, ldkv, Mq, L, H, out, ldo, part, part_bytes, stream,
                                   timing_name);
}

}  // namespace echo

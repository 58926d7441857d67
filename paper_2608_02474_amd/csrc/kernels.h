// Launchers of the gfx950 kernels, shared by the kernel files and the C ABI.
// Every launcher enqueues on `stream` and returns the launch error.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace echo {

typedef uint16_t bf16_t;

enum GemmEpi { EPI_BIAS = 0, EPI_GELU = 1, EPI_GATE_RES = 2 };

// C[m, n] = epilogue(sum_k A[row(m), k] B[n, k] + bias[n]), see gemm_bf16.hip.
struct GemmBf16Args {
  const bf16_t* A;
  int64_t lda;
  const int32_t* a_rows;    // optional: A row of output row m is a_rows[m]
  int64_t a_nrows;          // rows of A (every row index is below it)
  const bf16_t* B0;
  const bf16_t* B1;         // rows n >= n_split come from B1 (row n - n_split)
  int n_split;
  int64_t ldb;
  const bf16_t* bias0;
  const bf16_t* bias1;
  int M, N, K;
  void* C;                  // bf16 (EPI_BIAS, EPI_GELU) or fp32 (EPI_GATE_RES)
  int64_t ldc;
  const float* gate;        // [N], EPI_GATE_RES
  const void* res;          // EPI_GATE_RES residual rows (bf16 or fp32)
  int64_t ldr;
  const int32_t* res_rows;  // optional gather of residual rows
  int res_bf16;
  float* part;              // optional: fp32 partial tiles of the split-K tail
  size_t part_bytes;
  // set by the launcher: the first split tile, k splits per split tile (<= 1:
  // none), k-steps per split, and the workgroups that run split pieces (the
  // first npieces of the launch; the rest run whole tiles from tile 0)
  int tile_base, nsplit, kps;
  int npieces;
};

struct GemmF32Args {
  const float* A;
  int64_t lda;
  const int32_t* a_rows;
  const float* B0;
  const float* B1;
  int n_split;
  int64_t ldb;
  const float* bias0;
  const float* bias1;
  int M, N, K;
  float* C;
  int64_t ldc;
  const float* gate;
  const float* res;
  int64_t ldr;
  const int32_t* res_rows;
};

hipError_t launch_energy(const float* audio, int64_t n_samples, int T, int sr, int n_fft, int hop,
                         int n_bands, float* band_energy, float* frame_energy, float* frame_weight,
                         double* part, double* e_scratch, hipStream_t stream);
int energy_max_frames(int64_t n_samples, int T, int n_fft, int hop);

hipError_t launch_select(int dtype_bf16, const void* x, const void* xref, const float* fw, int L, int N,
                         int D, double xi, int k, int threshold_mode, float threshold, float* s,
                         double* num, double* den, int32_t* idx, uint8_t* mask, int32_t* n_sel,
                         double* step_delta, hipStream_t stream);

hipError_t launch_saliency(int dtype_bf16, const void* x, const void* xref, const float* fw, int L, int N,
                           int D, double xi, float* s, double* num, double* den, double* step_delta,
                           hipStream_t stream);
// with step_delta set, a second workgroup of the same launch writes the
// step-level sum of num / den (the saliency pass's by-products)
hipError_t launch_topk(const float* s, int L, int k, int threshold_mode, float threshold, int32_t* idx,
                       uint8_t* mask, int32_t* n_sel, hipStream_t stream, const double* num = nullptr,
                       const double* den = nullptr, double xi = 0.0, double* step_delta = nullptr);

// two-stage selection (anchor segments, then min(k, N) tokens per anchor)
hipError_t launch_topk_segments(const float* s, const uint8_t* anchors, int T, int N, int k, int32_t* idx,
                                uint8_t* mask, int32_t* n_sel, hipStream_t stream);
// anchor segments: mode 0 top-k of keys, mode 1 evenly spaced; T <= max_anchor_segments()
hipError_t launch_anchors(const float* keys, int T, int k, int mode, uint8_t* anchors, hipStream_t stream);
int max_anchor_segments();

hipError_t launch_cache_update(int dtype_bf16, const void* x, const int32_t* idx, const uint8_t* mask,
                               int n_sel, int L, int D, const float* y_sel, void* xref, int8_t* codes,
                               float* scale, void* y, hipStream_t stream);

// codec 0: int8 residual against xref (launch_cache_update); 1: the output in
// the activation dtype in `store`; 2: int8 codes of the output itself
hipError_t launch_cache_codec(int dtype_bf16, int codec, const void* x, const int32_t* idx,
                              const uint8_t* mask, int n_sel, int L, int D, const float* y_sel, void* xref,
                              void* store, int8_t* codes, float* scale, void* y, hipStream_t stream);

hipError_t launch_refcache_init(int L, int n_chains, int capacity, int32_t* refcount, int32_t* free_list,
                                int32_t* free_top, int32_t* chain_ref, int32_t* ent_slot, uint8_t* ent_kind,
                                float* scale, hipStream_t stream);
hipError_t launch_refcache_update(int dtype_bf16, const void* x, const int32_t* idx, const uint8_t* mask,
                                  int n_sel, int L, int D, int chain_len, float tau, const float* y_sel,
                                  void* pool, int32_t* refcount, int32_t* free_list, int32_t* free_top,
                                  int32_t* chain_ref, int32_t* ent_slot, uint8_t* ent_kind, int8_t* codes,
                                  float* scale, void* xref, void* y, hipStream_t stream);

// Wan-style block extras: rotary table ((cos, sin) per axis position and pair),
// in-place qk RMSNorm (+ 3D RoPE when tab is not null) of M rows of z, and
// out = (a ? a : 0) + beta
int rope_table_entries(int T, int gh, int gw, int dh);
hipError_t launch_rope_table(int T, int gh, int gw, int dh, double base, float2* tab, hipStream_t stream);
hipError_t launch_qk_norm_rope(bf16_t* z, int64_t ldz, int M, int D, const float* g, float eps,
                               const int32_t* rows, const float2* tab, int L, int T, int gh, int gw, int dh,
                               hipStream_t stream);
hipError_t launch_vec_shift(const float* a, float beta, float* out, int n, hipStream_t stream);

hipError_t launch_modln_input(int dtype_bf16, const void* x, int M, int D, const float* shift,
                              const float* scale, float eps, void* out, hipStream_t stream);
hipError_t launch_modln_x1(int dtype_bf16, const float* x1, int M, int D, const float* shift,
                           const float* scale, float eps, void* out, hipStream_t stream);

hipError_t launch_gemm_bf16(const char* name, int epi, const GemmBf16Args& a, hipStream_t stream);
hipError_t launch_gemm_f32(const char* name, int epi, const GemmF32Args& a, hipStream_t stream);

// `part` (part_bytes; attn_partial_bytes(Mq_max, L, H) is enough for any Mq
// up to Mq_max) holds the partial results of the key-range pieces that
// balance the last round; with part == nullptr, or less room, every work item
// runs whole.
hipError_t launch_attn_bf16(const bf16_t* q, int64_t ldq, const bf16_t* k, const bf16_t* v,
                            int64_t ldkv, int Mq, int L, int H, bf16_t* out, int64_t ldo,
                            float* part, size_t part_bytes, hipStream_t stream,
                            const char* timing_name = "attn_fwd_bf16");
size_t attn_partial_bytes(int Mq_max, int L, int H);
// bytes that hold the partial results of the GEMMs' split tails (256 fp32
// tiles of 256 x 256)
size_t gemm_partial_bytes();
// compute units of the current device (cached; 256 if the query fails)
int device_cu_count();
// sustained rate of a bf16 MFMA stream (pattern 0: attention, 1: GEMM; gaussian 0/1), TFLOP/s
hipError_t run_mfma_ceiling(int pattern, int gaussian, double seconds, double* tflops, hipStream_t stream);
hipError_t launch_attn_f32(const float* q, int64_t ldq, const float* k, const float* v, int64_t ldkv,
                           int Mq, int L, int H, int dh, float* out, int64_t ldo, hipStream_t stream);

}  // namespace echo

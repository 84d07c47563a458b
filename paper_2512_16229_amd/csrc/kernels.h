// Host-side launchers of the gfx950 kernels (internal to liblopa).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lopa.h"

// ----------------------------------------------------------- step kernels
// Positions [0, n_elig) (1 <= n_elig <= L <= 256) are eligible for the Eq. 1
// fallback and the lookahead fills.
hipError_t launch_build_branches(const int32_t* tokens, const float* conf, const int32_t* pred,
                                 int L, int n_elig, int mask_id, float tau, int k,
                                 int32_t* branch_tokens, int32_t* fill_pos, uint8_t* valid,
                                 int32_t* n_valid, hipStream_t s);
// metric 0: Eq. 2 mean; 1: window minimum (window >= 1); 2: lowest-segment
// mean (0 < eta <= 1). nb <= 1024, L <= 256.
hipError_t launch_select(const int32_t* bt, const float* conf, const int32_t* pred,
                         const uint8_t* valid, int nb, int L, int mask_id, int metric,
                         int window, float eta, float* scores, int32_t* winner, int32_t* nt,
                         float* nc, int32_t* np, int32_t* nu, hipStream_t s);
// KV layouts. Cache: [layers][2][Hkv][d * vld] (vld = max_len rounded up to
// 32); each head's K and V region in the KV tile layout of common.h
// (kv_k_off / kv_v_off). Staging: [branches][layers][2][Hkv][d * vlds], the
// same with Lcap rounded up to 32.
hipError_t launch_commit(const uint16_t* staging, uint16_t* cache, const int32_t* winner,
                         int nb_last, int layers, int Hkv, int vlds, int vld, int d, int P,
                         int L, int32_t* append_offset, hipStream_t s);
// Copy positions of one layer between the cache (or staging) and a caller
// buffer [Hkv][len][d] for K and V. to_cache: caller -> cache. head_stride:
// elements between heads of the cache side; ld: positions a head region holds
// (a multiple of 32; start + len <= ld).
hipError_t launch_kv_rows(uint16_t* cache_k, uint16_t* cache_v, int64_t head_stride, int ld,
                          int Hkv, int d, int start, int len, uint16_t* buf_k, uint16_t* buf_v,
                          int to_cache, hipStream_t s);
// Multi-block window (lopa_window in device memory; see step_kernels.hip):
// the header of a new window; the gates after a selection (tokens / conf /
// pred: the window rows, capacity w_max * L <= 256; out: the generated
// tokens); the commit of the blocks the last update moved out (rows [0, n) of
// the winner's staging of the last verify forward, n <= last_L).
hipError_t launch_window_init(lopa_window* win, int L, int w_max, int n_blocks, int prefix_len,
                              int mask_id, int add_min, int act_min, hipStream_t s);
hipError_t launch_window_update(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred,
                                int32_t* out, hipStream_t s);
hipError_t launch_window_commit(const uint16_t* staging, uint16_t* cache, const int32_t* winner,
                                lopa_window* win, int nb_last, int last_L, int max_len,
                                int layers, int Hkv, int vlds, int vld, int d, hipStream_t s);

// ------------------------------------------------------------ weight repack
// Pack the rows of up to three [rows_i, K] bf16 sources (stacked in order) into
// the GEMM weight layout: 16-row blocks grouped in tiles of nb blocks, stored
// [tile][KC][nb][2][64 lanes][8] (one 1 KiB B-operand fragment per (block,
// 64-column chunk, 32-column half)), so that one GEMM iteration streams one
// contiguous nb x 2 KiB chunk and a tile's k-range is one contiguous run.
// `blocks` (a multiple of nb) blocks are written; rows past the sources are
// zero. pairs: block 2p holds rows [16p, 16p + 16) of source 0 and block 2p + 1
// the same rows of source 1 (gate / up pairing for the SwiGLU epilogue).
// K: source row length; KP (a multiple of 256, >= K): packed width, zero-filled.
hipError_t launch_repack(const uint16_t* s0, int r0, const uint16_t* s1, int r1,
                         const uint16_t* s2, int r2, int K, int KP, int blocks, int nb, int pairs,
                         uint16_t* dst, hipStream_t s);
hipError_t launch_bf16_to_f32(const uint16_t* src, float* dst, int n, hipStream_t s);
// bytes [0, bytes) of device memory p set to zero by a kernel (p and bytes
// multiples of 16)
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);

// ---------------------------------------------------------------- per-row
// x[r] = embed[tokens[r]] (fp32) and a[r] = pack(rmsnorm(x[r]) * w) for r < M.
hipError_t launch_embed_norm(const int32_t* tokens, const uint16_t* embed, int vocab,
                             const float* w, float eps, int M, int Mp, int H, float* x,
                             uint16_t* a, hipStream_t s);
// x[r] += sum over s < S of part[s][r] (row-major [S][Mp][H]; S = 0: none),
// then a[r] = pack(rmsnorm(x[r]) * w), for r < M. H % 256 == 0.
hipError_t launch_resnorm(const float* part, int S, const float* w, float eps, int M, int Mp,
                          int H, float* x, uint16_t* a, hipStream_t s);
// FP8 (E4M3, per-row scale) forms: launch_resnorm with the normed row written
// as the packed FP8 operand a8 and its scale sa[r]; the packed bf16 operand a
// (K columns) requantised to FP8; per-row scaling pairs of a bf16 weight
// [rows][K]; the FP8 weight repack (see gemm.hip; KP % 512 == 0)
hipError_t launch_resnorm8(const float* part, int S, const float* w, float eps, int M, int Mp,
                           int H, float* x, uint8_t* a8, float* sa, uint32_t* rowmax_zero,
                           hipStream_t s);
hipError_t launch_quant_rows8(const uint16_t* a, int K, int M, int Mp, const uint32_t* rowmax,
                              uint8_t* a8, float* sa, hipStream_t s);
hipError_t launch_rowscale(const uint16_t* w, int rows, int K, float* inv, float* scale,
                           hipStream_t s);
hipError_t launch_repack8(const uint16_t* s0, const float* inv0, const float* sc0, int r0,
                          const uint16_t* s1, const float* inv1, const float* sc1, int r1,
                          const uint16_t* s2, const float* inv2, const float* sc2, int r2, int K,
                          int KP, int blocks, int nb, int pairs, uint8_t* dst, float* sw,
                          hipStream_t s);
hipError_t launch_embed_norm8(const int32_t* tokens, const uint16_t* embed, int vocab,
                              const float* w, float eps, int M, int Mp, int H, float* x,
                              uint8_t* a8, float* sa, uint32_t* rowmax_zero, hipStream_t s);
// merge per-tile softmax partials into conf / pred
hipError_t launch_lm_merge(const float* pm, const float* ps, const int32_t* pi, int M,
                           int tiles, float* conf, int32_t* pred, hipStream_t s);

// ---------------------------------------------------------------- GEMM
enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LMHEAD = 3 };
// most k-splits of the QKV projection (its fix-up sums them with the count as a constant)
constexpr int QKV_MAX_SPLITS = 8;

struct GemmArgs {
  const uint16_t* A;   // packed activations, Mp rows, K columns
  const uint16_t* W;   // packed weights [tiles][KC][nb blocks of 16 columns][2][64][8]
  int M, Mp, N, KC;    // KC = K / 64 iterations per tile, a multiple of 4
  int nb;              // 16-column blocks per tile (an instantiated width)
  int tiles;           // column tiles
  int splits;          // k-splits per tile; > 1: partial sums + fix-up kernel
  int mtiles;          // row tiles of 256 rows; Mp = 256 * mtiles
  int gcols;           // workgroups per row tile (tiles * splits when splits > 1)
  float* partials;     // EPI_QKV: [mtiles][tiles][splits][4 waves][4][nb][64][4] fp32;
                       // EPI_RESID (splits > 1): row-major [splits][Mp][N] fp32, added by
                       // the following launch_resnorm (no fix-up kernel)
  // EPI_QKV
  const float* bias;   // [N] or null
  const float* rope;   // [max_pos][d/2][2] (cos, sin)
  uint16_t* q_out;     // [nb][Hq][L][d]
  uint16_t* staging;   // [nb][layers][2][Hkv][d * vlds] (the KV tile layout)
  int layer, layers, Hq, Hkv, d, L, P;
  int vlds;            // staging V leading dimension
  // EPI_RESID
  float* x;            // [M][N] fp32 residual stream (row stride N)
  // EPI_SWIGLU
  uint16_t* a_out;     // packed, Mp rows, N/2 columns
  // EPI_LMHEAD
  float* pm;           // [M][tiles] running max
  float* ps;           // [M][tiles] sum of exp(l - max)
  int32_t* pi;         // [M][tiles] argmax
  int vocab, mask_id;
  // FP8 operands (f8 != 0; any epilogue): A and W hold E4M3 bytes in
  // the same fragment layout (a 16-byte lane slot holds 16 values of K instead
  // of 8), KC counts 128-wide k-chunks, and the epilogue scales the fp32 sum
  // of products by sa[row] * sw[packed column]
  int f8;
  // rot != 0: each workgroup starts its k-range at chunk 4 (column tile mod
  // quads) and wraps, so the workgroups of an XCD, which otherwise advance in
  // step, read different slices of the shared activation operand at a time
  // (spread over the L2 channels); the sums of a column stay in one fixed order
  int rot;
  const float* sa;     // [Mp] per-row activation scales
  const float* sw;     // [blocks * 16] per-column weight scales, packed column order
  uint32_t* rowmax;    // FP8 EPI_SWIGLU: atomic maximum of |output| (float bits) per row,
                       // zeroed beforehand (the requantisation's row scale)
};
// bytes of LDS of gemm_kernel<epi, nb> (-1: not instantiated)
int gemm_smem_bytes(int epi, int nb);
hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  const uint16_t* q;       // [nb][Hq][L][d] bf16 (post-RoPE)
  const uint16_t* kcache;  // layer's K cache, heads d * vld apart (KV tile layout)
  const uint16_t* vcache;  // layer's V cache, heads d * vld apart (KV tile layout)
  const uint16_t* staging; // [nb][layers][2][Hkv][d * vlds]
  uint16_t* out;           // packed activations (Mp rows, Hq*d columns)
  int nb, L, P, Hq, Hkv, d, vld, layer, layers, vlds, Mp;
  float scale;
  // block-causal mask inside the block (cblk > 0, a multiple of 16 dividing L):
  // a row of sub-block r / cblk sees the prefix and the block keys of the
  // sub-blocks up to its own. 0: full attention inside the block.
  int cblk;
  // working memory of the grouped form for long key ranges (per key split:
  // row maxima, sums and partial outputs); null or too small: not used
  float* scratch;
  size_t scratch_bytes;
  // non-null: the largest |value| of each output row (over all heads, of the
  // stored bf16 values) merged into rowmax[row] as float bits by an atomic
  // unsigned maximum (order-free; zeroed beforehand): the row scales of the
  // FP8 output projection
  uint32_t* rowmax;
};
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);
// bytes of AttnArgs::scratch that let the grouped form run with its full key
// splits for nb branches of L rows at any prefix (0: the shape never takes it)
size_t attention_scratch_bytes(int nb, int L, int Hq, int Hkv, int d);

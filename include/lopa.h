/*
 * lopa.h - C ABI of an MI355X (gfx950) implementation of the per-iteration
 * branch-verification step of LoPA, Lookahead Parallel Decoding for diffusion
 * LLMs (arXiv 2512.16229).
 *
 * One LoPA iteration (Alg. 1) on one GPU is four calls, all enqueued on the
 * caller's HIP stream, with no host synchronisation inside a step:
 *
 *   lopa_build_branches            Eq. 1 anchor fill + top-k lookahead branches
 *                                  (Alg. 1 steps 1-2)
 *   lopa_verify_forward            one batched forward of all k+1 branches of
 *                                  the active block against the shared-prefix
 *                                  KV cache; per-position Conf and candidate
 *                                  (Alg. 1 step 3, Sec. 3.1, Sec. 3.3)
 *   lopa_branch_confidence_select  Eq. 2 branch confidence, B* = argmax, and the
 *                                  next state taken from B*'s verification
 *                                  outputs (logit reuse, Sec. 3.2)
 *   lopa_commit_kv                 write B*'s block K/V into the static cache
 *                                  (single-GPU form of the Pre-Write /
 *                                  Commit-Winner-Cache protocol, Sec. 3.4)
 *
 * Conventions for every call:
 *   - All array arguments are DEVICE pointers unless stated otherwise; the
 *     caller owns them. The library owns handles, repacked weights, the KV
 *     cache, the per-branch K/V staging and its workspace.
 *   - `stream` is a hipStream_t (NULL = the default stream). Outputs are valid
 *     in stream order after the call; nothing here synchronises the host.
 *   - Return value: LOPA_OK (0) or a negative status. Argument checks run on
 *     the host before any HIP call, so invalid arguments never reach the GPU.
 *     lopa_last_error() returns a message for the calling thread's last error.
 *   - No call allocates device memory except lopa_model_create and
 *     lopa_kv_create.
 *   - Calls that share a lopa_kv must be ordered on one stream; concurrent
 *     verify_forward calls on one lopa_kv race on its workspace.
 */
#ifndef LOPA_H
#define LOPA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  LOPA_OK = 0,
  LOPA_EINVAL = -1,    /* null pointer, k < 0, tau outside [0, 1], bad config  */
  LOPA_ESHAPE = -2,    /* L, n_branches or a model dimension the kernels do   */
                       /* not support, or larger than the lopa_kv capacity    */
  LOPA_ECAPACITY = -3, /* prefix_len + L > max_len of the cache               */
  LOPA_EHIP = -4,      /* a HIP call failed; the message names the hipError_t */
  LOPA_ENOMEM = -5     /* device allocation failed                            */
};

/* Largest supported values (checked by the calls). */
#define LOPA_MAX_BLOCK 256   /* L: positions of the active block (window)   */
#define LOPA_MAX_ROWS 2048   /* n_branches * L rows in one verify forward   */
#define LOPA_WINDOW_MAX_BLOCKS 16  /* blocks of a multi-block window        */

/* Decoder shape (Qwen2.5 / LLaMA-style pre-norm decoder, the layout of the
 * paper's Dream-7B / DiffuCoder-7B backbones; the paper names only the
 * models). Constraints: hidden % 256 == 0, head_dim in {64, 128},
 * heads % kv_heads == 0, heads * head_dim == hidden, ffn % 64 == 0,
 * 0 <= mask_id < vocab. */
typedef struct lopa_model_cfg {
  int32_t layers;
  int32_t hidden;
  int32_t heads;      /* query heads                     */
  int32_t kv_heads;   /* key/value heads (grouped query) */
  int32_t head_dim;
  int32_t ffn;        /* SwiGLU intermediate size        */
  int32_t vocab;
  int32_t mask_id;    /* the mask token: position unfilled <=> token == mask_id */
  float rms_eps;
  float rope_theta;   /* rotate-half RoPE base            */
  int32_t qkv_bias;   /* 1: q/k/v projections have biases */
} lopa_model_cfg;

/* One layer's weights: bf16 DEVICE arrays in PyTorch [out, in] row-major
 * layout. They are only read during lopa_model_create (repacked into library
 * buffers); the caller may free them afterwards. */
typedef struct lopa_layer_weights {
  const void* wq;      /* [heads*head_dim, hidden]    */
  const void* wk;      /* [kv_heads*head_dim, hidden] */
  const void* wv;      /* [kv_heads*head_dim, hidden] */
  const void* bq;      /* [heads*head_dim] or NULL when qkv_bias == 0 */
  const void* bk;      /* [kv_heads*head_dim] or NULL */
  const void* bv;      /* [kv_heads*head_dim] or NULL */
  const void* wo;      /* [hidden, heads*head_dim]    */
  const void* w_gate;  /* [ffn, hidden]               */
  const void* w_up;    /* [ffn, hidden]               */
  const void* w_down;  /* [hidden, ffn]               */
  const void* ln1;     /* [hidden] pre-attention RMSNorm weight */
  const void* ln2;     /* [hidden] pre-MLP RMSNorm weight       */
} lopa_layer_weights;

typedef struct lopa_weight_ptrs {
  const void* embed;                 /* [vocab, hidden] bf16 device          */
  const lopa_layer_weights* layers;  /* HOST array of cfg.layers entries     */
  const void* final_norm;            /* [hidden] bf16 device                 */
  const void* lm_head;               /* [vocab, hidden] bf16 device, untied  */
} lopa_weight_ptrs;

typedef struct lopa_model lopa_model;
typedef struct lopa_kv lopa_kv;

/* ------------------------------------------------------------- lifecycle */

/* Validate cfg, allocate library buffers on the current device, repack the
 * weights on `stream` and wait for that to finish. *out receives the handle. */
int lopa_model_create(const lopa_model_cfg* cfg, const lopa_weight_ptrs* w,
                      void* stream, lopa_model** out);

/* Precision of the projections of a model (lopa_model_create_ex).
 * LOPA_PRECISION_BF16: every weight and GEMM operand bf16 (lopa_model_create).
 * LOPA_PRECISION_FP8_MLP: the three MLP projections (gate, up, down: three
 * quarters of a layer's weight bytes at the Dream-7B shape) in W8A8 FP8, the
 * paper's Ascend system's weight / activation quantisation (Sec. 3.4) carried
 * to the MI355X matrix cores: E4M3 values (no infinities, largest 448, round
 * to nearest even, saturating) with one fp32 scale per weight output channel
 * (max |w| / 448 of the row) and one per activation row (max |a| / 448 of the
 * row, computed where the row is produced: the RMSNorm for gate/up, a
 * requantisation of the bf16 SwiGLU output for down); the products are summed
 * in fp32 and the scales applied after the sum. Attention, QKV / O and the LM
 * head stay bf16. The caller's weights are still bf16.
 * LOPA_PRECISION_FP8: as FP8_MLP, and every other projection in W8A8 FP8 with
 * the same rules: QKV and the LM head (their activation rows are RMSNorm
 * outputs, so the norm writes the E4M3 rows and scales) and the output
 * projection (its activation rows are the bf16 attention output, quantised
 * with one scale per row over all heads by one more pass over them); the
 * attention itself stays bf16. */
enum { LOPA_PRECISION_BF16 = 0, LOPA_PRECISION_FP8_MLP = 1, LOPA_PRECISION_FP8 = 2 };
int lopa_model_create_ex(const lopa_model_cfg* cfg, const lopa_weight_ptrs* weights,
                         int32_t precision, void* stream, lopa_model** out);
void lopa_model_destroy(lopa_model* m);

/* Static KV cache of max_len positions for one sequence (Sec. 3.4: a
 * pre-allocated static cache instead of dynamic objects), plus K/V staging for
 * max_branches branches of a block of up to max_block positions, plus the
 * verify workspace. Cache layout (bf16, library-owned; read and write rows
 * through lopa_kv_read / lopa_kv_write, which use [kv_heads][len][head_dim]
 * whatever the internal layout): layers outermost, then K / V, then KV heads;
 * each head's K region and V region hold tiles of 32 consecutive positions
 * (max_len rounded up to 32), head_dim x 32 values per tile, stored in the
 * order the attention kernels' matrix-core instructions take them: every
 * 1 KiB operand fragment (K: 16 positions x 32 dimensions; V: 16 dimensions x
 * 32 positions) is one contiguous run, 16 bytes per lane of a wavefront. The
 * per-branch staging has the same layout with max_block. Zero-initialised. */
int lopa_kv_create(const lopa_model* m, int32_t max_len, int32_t max_branches,
                   int32_t max_block, lopa_kv** out);
void lopa_kv_destroy(lopa_kv* kv);

const char* lopa_strerror(int status);
const char* lopa_last_error(void);

/* ----------------------------------------------------------- hot path */

/* Alg. 1 steps 1-2 (Eq. 1; Sec. 3.2 "Look ahead Multiple TFOs in Parallel").
 * In:  tokens[L] int32 (the block; position i unfilled <=> tokens[i] == mask_id,
 *      at least one must be unfilled), conf[L] float32 and pred[L] int32 from
 *      the forward pass on exactly these tokens (values at filled positions are
 *      ignored), tau in [0, 1], k >= 0.
 * Anchor B0: I_fill = {unfilled i : conf[i] > tau} (strict), or, if empty, the
 *      single unfilled position of largest conf (lowest position on ties);
 *      B0 = tokens with pred written at I_fill.
 * Lookahead: the k_eff = min(k, |M_B0|) unfilled positions of B0 with the
 *      largest conf (ties: lower position first); branch j (1..k_eff) is B0
 *      with position p_j also set to pred[p_j].
 * Out: branch_tokens[(k+1)*L] int32, branch-major (row j = B_j); rows
 *      j > k_eff are copies of B0. fill_pos[k+1] int32 (-1 for B0 and padding,
 *      else p_j). valid[k+1] uint8 (1 for j <= k_eff). n_valid[1] int32 =
 *      1 + k_eff. One workgroup; L <= LOPA_MAX_BLOCK. */
int lopa_build_branches(const int32_t* tokens, const float* conf, const int32_t* pred,
                        int32_t L, int32_t mask_id, float tau, int32_t k,
                        int32_t* branch_tokens, int32_t* fill_pos, uint8_t* valid,
                        int32_t* n_valid, void* stream);

/* The same over a multi-block window (Sec. 3.3, integration with D2F: all
 * active blocks form one window for branch exploration). tokens / conf / pred
 * cover the L window positions; positions [0, n_eligible) are those of the
 * fully activated blocks (a prefix of the window, 1 <= n_eligible <= L). The
 * Eq. 1 threshold fill uses every unfilled position; the argmax fallback and
 * the k lookahead positions are taken among the eligible ones only (at least
 * one eligible position must be unfilled). n_eligible = L is
 * lopa_build_branches. Errors as lopa_build_branches, and LOPA_EINVAL for
 * n_eligible outside [1, L]. */
int lopa_build_branches_window(const int32_t* tokens, const float* conf, const int32_t* pred,
                               int32_t L, int32_t n_eligible, int32_t mask_id, float tau,
                               int32_t k, int32_t* branch_tokens, int32_t* fill_pos,
                               uint8_t* valid, int32_t* n_valid, void* stream);

/* Alg. 1 step 3 "single pass" + Sec. 3.1 Conf + Sec. 3.3 attention pattern.
 * In:  branch_tokens[n_branches*L] int32 (block rows at positions
 *      prefix_len .. prefix_len+L-1), the cache rows [0, prefix_len).
 * Attention: each row sees all prefix_len committed positions and all L rows
 *      of its own branch (full attention inside the block); branches do not
 *      see each other.
 * Out: conf[n_branches*L] float32 = the largest probability of the softmax over
 *      the vocabulary with mask_id excluded; pred[n_branches*L] int32 = its
 *      token (lowest id on ties). Both are produced for every row.
 *      The post-RoPE K and V of every branch's block rows go to the lopa_kv's
 *      staging (all layers), ready for lopa_commit_kv.
 * Compute: bf16 weights and GEMM inputs, fp32 accumulation, fp32 residual
 *      stream, norms, RoPE, softmax and logits.
 * Limits: n_branches <= max_branches, L <= max_block of the lopa_kv,
 *      n_branches*L <= LOPA_MAX_ROWS; prefix_len + L <= max_len. */
int lopa_verify_forward(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                        const int32_t* branch_tokens, int32_t n_branches, int32_t L,
                        float* conf, int32_t* pred, void* stream);

/* Eq. 2 and Alg. 1 step 3 selection; Sec. 3.2 logit reuse.
 * In:  branch_tokens[n_branches*L], conf/pred[n_branches*L] from
 *      lopa_verify_forward on those branches, valid[n_branches].
 * scores[j] = mean of conf over row j's positions holding mask_id (Eq. 2),
 *      +inf if the row has none, -inf if valid[j] == 0.
 * winner[0] = argmax_j scores[j] (lowest j on ties).
 * next_tokens/next_conf/next_pred[L] = row winner of the inputs (the state of
 *      the next iteration); next_unfilled[0] = number of mask_id positions in
 *      it (0 = block complete). One workgroup. */
int lopa_branch_confidence_select(const int32_t* branch_tokens, const float* conf,
                                  const int32_t* pred, const uint8_t* valid,
                                  int32_t n_branches, int32_t L, int32_t mask_id,
                                  float* scores, int32_t* winner, int32_t* next_tokens,
                                  float* next_conf, int32_t* next_pred,
                                  int32_t* next_unfilled, void* stream);

/* Alternative branch confidences (Sec. 3.2 names them after Eq. 2 without a
 * formula; these are the readings implemented). Same arguments, outputs and
 * selection rule as lopa_branch_confidence_select, with scores[j] for a valid
 * row j with m > 0 unfilled positions p_1 < ... < p_m, c_i = conf[j][p_i]:
 *   LOPA_METRIC_MEAN            the Eq. 2 mean (window, eta unused);
 *   LOPA_METRIC_WINDOW_MIN      the smallest mean of `window` consecutive c_i
 *                               ("local quality"; the mean of all m if
 *                               m <= window); window >= 1;
 *   LOPA_METRIC_LOWEST_SEGMENT  the mean of the ceil(eta*m) smallest c_i, at
 *                               least one ("weak links"; ceil of the double
 *                               product of eta and m); 0 < eta <= 1.
 * m = 0 gives +inf and an invalid row -inf, as in Eq. 2. Errors: LOPA_EINVAL
 * for an unknown metric or a parameter outside its range. */
enum { LOPA_METRIC_MEAN = 0, LOPA_METRIC_WINDOW_MIN = 1, LOPA_METRIC_LOWEST_SEGMENT = 2 };
int lopa_branch_confidence_select_metric(const int32_t* branch_tokens, const float* conf,
                                         const int32_t* pred, const uint8_t* valid,
                                         int32_t n_branches, int32_t L, int32_t mask_id,
                                         int32_t metric, int32_t window, float eta, float* scores,
                                         int32_t* winner, int32_t* next_tokens, float* next_conf,
                                         int32_t* next_pred, int32_t* next_unfilled,
                                         void* stream);

/* Sec. 3.4 Commit-Winner-Cache, single-GPU form: copy the staged post-RoPE
 * K/V of branch *winner (a DEVICE int32, read by the kernel: no host sync) for
 * all layers into cache rows [prefix_len, prefix_len + L). The staging must
 * come from the last lopa_verify_forward on this lopa_kv with the same
 * prefix_len and L. append_offset[0] (device int32) receives prefix_len.
 * A winner outside [0, n_branches of that forward) writes nothing and sets
 * append_offset[0] = -1. */
int lopa_commit_kv(lopa_kv* kv, const int32_t* winner, int32_t prefix_len, int32_t L,
                   int32_t* append_offset, void* stream);

/* Commit only the first n_rows (1 <= n_rows <= L) staged positions of the
 * winner: cache rows [prefix_len, prefix_len + n_rows). For a multi-block
 * window (Sec. 3.3) whose first block has been filled: that block leaves the
 * window and its K/V enter the prefix, while the later blocks stay active.
 * prefix_len and L must be those of the last lopa_verify_forward (the window
 * length); otherwise as lopa_commit_kv. */
int lopa_commit_kv_rows(lopa_kv* kv, const int32_t* winner, int32_t prefix_len, int32_t L,
                        int32_t n_rows, int32_t* append_offset, void* stream);

/* -------------------------------------------- multi-block window (D2F) */

/* Sec. 3.3, integration with D2F: the active blocks form one window whose
 * positions are explored together, blocks join the window by the tau_add gate
 * and become fully activated by the tau_act gate, and a completed leading
 * block leaves it (its K/V enter the prefix). The window's state lives in
 * device memory in this struct (caller-allocated, device); the three calls
 * below read and write it on the stream, so the gates need no host copy of the
 * window. A host loop reads the first words (blocks, eligible, prefix_len,
 * need_initial, done) once per iteration: the next iteration's launch shapes
 * depend on them. Gates in the library's readings (tau as fractions of a
 * block's L positions, compared in double on the host and kept as counts):
 *   - an empty window with blocks left opens one, fully activated, with
 *     need_initial = 1 (its initial forward, one branch over its L rows, has
 *     not run); then blocks are appended, not activated, while the window has
 *     fewer than w_max blocks, blocks remain, and the last block has at least
 *     add_min = ceil(tau_add L) filled positions;
 *   - after a selection (lopa_window_update): block b >= 1 becomes fully
 *     activated when block b - 1 is and has at least act_min = ceil(tau_act L)
 *     filled positions (block order); the leading blocks with no masked
 *     position leave the window (tokens to the output, K/V committed by
 *     lopa_window_commit), the rest moves to the front with its new first
 *     block fully activated; then the opening / appending above.
 * Opened and appended blocks hold mask_id, conf 0 and pred mask_id. */
typedef struct lopa_window {
  int32_t blocks;          /* blocks in the window (its length is blocks * L)       */
  int32_t eligible;        /* positions of its fully activated leading blocks:       */
                           /* the n_eligible of lopa_build_branches_window          */
  int32_t prefix_len;      /* committed positions (the verify forwards' prefix_len) */
  int32_t need_initial;    /* 1: block 0 was just opened; run its initial forward    */
  int32_t done;            /* 1: all n_blocks blocks committed                      */
  int32_t added;           /* blocks opened or appended so far                      */
  int32_t committed;       /* blocks committed so far                               */
  int32_t last_commit;     /* blocks the last update moved out of the window        */
  int32_t last_commit_at;  /* the prefix_len they are committed at                  */
  int32_t error;           /* 1: lopa_window_commit found its inputs invalid        */
  int32_t L, w_max, n_blocks, mask_id, add_min, act_min;
  int32_t active[LOPA_WINDOW_MAX_BLOCKS];  /* 1: block fully activated               */
} lopa_window;

/* Start a window for n_blocks blocks of L positions after prefix_len committed
 * positions: writes the header and opens block 0 into tokens / conf / pred
 * (device, capacity w_max * L each) by the rules above. Host checks: null
 * pointers, 1 <= w_max <= LOPA_WINDOW_MAX_BLOCKS, w_max * L <= LOPA_MAX_BLOCK,
 * n_blocks >= 1, prefix_len >= 0, tau_add and tau_act in [0, 1] (LOPA_EINVAL /
 * LOPA_ESHAPE). */
int lopa_window_init(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred, int32_t L,
                     int32_t w_max, int32_t n_blocks, int32_t prefix_len, int32_t mask_id,
                     double tau_add, double tau_act, void* stream);

/* The gates after a selection: tokens / conf / pred (device) hold the winner's
 * window rows (the next_tokens / next_conf / next_pred of
 * lopa_branch_confidence_select over the window); they are updated in place
 * to the next window. Tokens of completed leading blocks are appended to
 * out_tokens (device, n_blocks * L int32, block order). */
int lopa_window_update(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred,
                       int32_t* out_tokens, void* stream);

/* Commit the K/V of the blocks the last lopa_window_update moved out of the
 * window: the first last_commit * L staged rows of branch *winner (device) of
 * the last lopa_verify_forward on kv (which must be that of the window's
 * iteration) go to cache rows [last_commit_at, ...). Nothing if none left.
 * The row count is read on the device: inputs that do not fit (winner outside
 * the forward's branches, more rows than it staged, past max_len) commit
 * nothing and set win->error = 1. */
int lopa_window_commit(lopa_kv* kv, const int32_t* winner, lopa_window* win, void* stream);

/* ---------------------------------------------------------- inspection */

/* Copy cache rows [start, start+len) of one layer to k_dst, v_dst (device,
 * bf16 [kv_heads][len][head_dim] each). For tests and checkpoints. */
int lopa_kv_read(const lopa_kv* kv, int32_t layer, int32_t start, int32_t len,
                 void* k_dst, void* v_dst, void* stream);

/* Write cache rows [start, start+len) of one layer from k_src, v_src (same
 * layout as lopa_kv_read). Restores a checkpointed prefix. */
int lopa_kv_write(lopa_kv* kv, int32_t layer, int32_t start, int32_t len,
                  const void* k_src, const void* v_src, void* stream);

/* Copy the staged block K/V of one branch and layer from the last
 * lopa_verify_forward to k_dst, v_dst (device, bf16 [kv_heads][L][head_dim]). */
int lopa_kv_read_staging(const lopa_kv* kv, int32_t branch, int32_t layer,
                         void* k_dst, void* v_dst, void* stream);

/* Attention mask inside the active block (window) of later verify forwards.
 * sub_block = 0 (the default): full attention among the block's L rows
 * (Sec. 3.3). sub_block = c > 0, a multiple of 16: the block-wise causal mask
 * of the paper's Ascend system (Sec. 3.4): the L rows are consecutive
 * sub-blocks of c rows (the window's blocks) and a row of sub-block b attends
 * to the committed prefix and to the rows of sub-blocks 0..b of its own
 * branch. A block's K/V then never depend on later blocks, so the K/V a
 * completed leading block leaves in the cache (lopa_commit_kv_rows) are final
 * without a separate winner commit protocol. A verify forward with L > c needs
 * L % c == 0 (LOPA_ESHAPE otherwise); L <= c is unmasked. sub_block negative or
 * not a multiple of 16: LOPA_EINVAL. Host only; applies to later calls. */
int lopa_kv_set_block_causal(lopa_kv* kv, int32_t sub_block);

/* Launch timing of lopa_verify_forward with HIP events on the call's stream.
 * kinds_mask selects which launches get an event pair (bit i = kind i below);
 * 0 turns timing off. Events between launches cost a few microseconds each. */
enum {
  LOPA_PROF_QKV = 0,     /* QKV projection + bias + RoPE + K/V staging  */
  LOPA_PROF_ATTN = 1,    /* block attention                              */
  LOPA_PROF_OPROJ = 2,   /* output projection + residual                 */
  LOPA_PROF_GATEUP = 3,  /* gate/up projection + SwiGLU                  */
  LOPA_PROF_DOWN = 4,    /* down projection + residual                   */
  LOPA_PROF_LMHEAD = 5,  /* LM head + per-tile softmax partials          */
  LOPA_PROF_NORM = 6,    /* embedding / RMSNorm row kernels              */
  LOPA_PROF_MERGE = 7,   /* softmax merge -> conf / pred                 */
  LOPA_PROF_KINDS = 8
};
int lopa_kv_profile(lopa_kv* kv, int32_t kinds_mask);

/* Wait for the recorded events, and return per kind the summed launch time in
 * milliseconds (total_ms[LOPA_PROF_KINDS], host) and the number of timed
 * launches (launches[LOPA_PROF_KINDS], host) since the last read; resets them. */
int lopa_kv_profile_read(lopa_kv* kv, double* total_ms, int64_t* launches);

/* Diagnostics of the verify forward: run the embedding and the first n_layers
 * decoder layers (0 <= n_layers <= cfg.layers) of lopa_verify_forward on the
 * same arguments and copy the fp32 residual stream [n_branches*L][hidden]
 * (row = branch * L + position) to x_out (device). K/V staging of those layers
 * is written as by lopa_verify_forward; conf / pred are not produced. */
int lopa_debug_hidden(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                      const int32_t* branch_tokens, int32_t n_branches, int32_t L,
                      int32_t n_layers, float* x_out, void* stream);

/* For callers that cannot allocate device memory where they run the step
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): lopa_verify_forward with the same arguments, outputs and errors,
 * whose working memory (residual stream, packed GEMM operands, queries,
 * split-K partial sums, LM-head statistics; the KV cache and staging stay in
 * kv) lives in one device array compiled into the library, of
 * LOPA_NOALLOC_MAX_BYTES per GPU, held by every GPU the library runs on until
 * the process ends. The call allocates nothing and frees nothing; it enqueues
 * a small fill kernel that zeroes the operands' padding columns, then the
 * forward. A shape whose working memory exceeds LOPA_NOALLOC_MAX_BYTES
 * (64 MiB: 256 rows of the Dream-7B or LLaDA-8B shape fit, 512 do not) is
 * LOPA_ESHAPE before anything is enqueued; the current device must be the
 * model's (LOPA_EINVAL). Every call on a GPU shares that GPU's array: calls
 * that overlap on one GPU (other streams or threads) race and give undefined
 * results; calls ordered on one stream do not. The first call on a device
 * looks up the array's address there (not inside a capture). */
#define LOPA_NOALLOC_MAX_BYTES (64ull << 20)
int lopa_verify_forward_noalloc(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                                const int32_t* branch_tokens, int32_t n_branches, int32_t L,
                                float* conf, int32_t* pred, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LOPA_H */

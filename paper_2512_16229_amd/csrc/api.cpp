// C ABI of liblopa: argument checks, handles, device buffers and the launch
// sequence of one verify forward. Every entry point validates its arguments on
// the host before touching the GPU and only enqueues work on the caller's
// stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/lopa.h"
#include "kernels.h"
#include "verify.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess) return fail(LOPA_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

struct DevBuf {
  void* p = nullptr;
  size_t n = 0;
};

int dalloc(DevBuf& b, size_t bytes, std::vector<void*>& owned) {
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(&b.p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(LOPA_ENOMEM, "hipMalloc(%zu bytes) failed: %s", bytes, hipGetErrorString(e));
  }
  b.n = bytes;
  owned.push_back(b.p);
  return LOPA_OK;
}

// Packed weights: [blocks of 16 output features][K / 64][2][64][8] bf16.
struct LayerPack {
  uint16_t* qkv;   // blk_qkv blocks, K = H (models with a bf16 QKV projection)
  uint16_t* o;     // blk_h blocks, K = Hq * d
  uint16_t* gu;    // blk_gu blocks (gate / up pairs), K = H (bf16 models)
  uint16_t* down;  // blk_h blocks, K = round256(F) (bf16 models)
  // FP8 MLP models: E4M3 weights (K = round512(H), round512(F)) and the scale
  // of every packed column
  uint8_t* gu8 = nullptr;
  uint8_t* down8 = nullptr;
  float* sw_gu = nullptr;
  float* sw_down = nullptr;
  // FP8 models: E4M3 QKV and output-projection weights (K = round512(H)) and
  // their column scales
  uint8_t* qkv8 = nullptr;
  float* sw_qkv = nullptr;
  uint8_t* o8 = nullptr;
  float* sw_o = nullptr;
  float* bias;     // [Nqkv] or null
  float* ln1;
  float* ln2;
};

// rows of the packed activation buffers: whole 256-row tiles
int padded_rows(int M) { return 256 * ((M + 255) / 256); }
int round256(int k) { return 256 * ((k + 255) / 256); }
int round512(int k) { return 512 * ((k + 511) / 512); }
int round_up(int x, int m) { return m * ((x + m - 1) / m); }

// Decomposition of one GEMM (see gemm.hip): tile width nb (16-column blocks)
// and k-splits S. SwiGLU and LM-head tiles are fixed (their epilogues need
// whole rows of a tile and no split); for the others the pair with the
// smallest estimated time is taken. Per round of workgroups the time is the
// larger of (a) the bytes one workgroup pulls into its CU (every k-chunk: the
// 256 x 64 bf16 activation chunk from L2 plus nb x 2 KiB of weights), at the
// per-CU rate measured for these kernels (~60 GB/s), and (b) the round's
// weight bytes at the sustained HBM rate (~6.5 TB/s); split-K adds its fp32
// partial sums, written (~5 TB/s) and read back by the small kernel that
// reduces them (~3 TB/s), and QKV its fix-up launch.
// The weights are packed per tile, so nb is chosen once, when the model is
// created (fixed_nb = 0: choose), and later plans choose S only.
struct GemmPlan {
  int nb, tiles, splits;
};
GemmPlan plan_gemm(int epi, int nblocks, int KC, int MT, int num_cu, int fixed_nb) {
  if (epi == EPI_SWIGLU) return {10, nblocks / 10, 1};
  if (epi == EPI_LMHEAD) return {fixed_nb, nblocks / fixed_nb, 1};
  constexpr double CU_BPUS = 60e3, HBM_BPUS = 6.5e6, PART_W_BPUS = 5e6, PART_R_BPUS = 3e6;
  constexpr double FIXUP_US = 7.0;
  const int Q = KC / 4;
  GemmPlan best{8, nblocks / 8, 1};
  double best_t = 1e300;
  for (int nb : {4, 8}) {
    if (fixed_nb && nb != fixed_nb) continue;
    const int tiles = nblocks / nb;
    for (int S = 1; S <= (epi == EPI_QKV ? std::min(Q, QKV_MAX_SPLITS) : Q); ++S) {
      const int64_t wgs = (int64_t)MT * tiles * S;
      const int64_t rounds = (wgs + num_cu - 1) / num_cu;
      const double iters = 4.0 * ((Q + S - 1) / S);
      const double per_cu = iters * (32768.0 + nb * 2048.0);
      const double w_round = (double)std::min<int64_t>(wgs, num_cu) * iters * nb * 2048.0;
      double t = (double)rounds * std::max(per_cu / CU_BPUS, w_round / HBM_BPUS);
      const double part = epi == EPI_QKV ? (double)wgs * nb * 16384.0
                                         : (S > 1 ? (double)S * MT * 256.0 * tiles * nb * 16 * 4 : 0.0);
      t += part / PART_W_BPUS + part / PART_R_BPUS;
      if (epi == EPI_QKV) t += FIXUP_US;
      if (t < best_t) {
        best_t = t;
        best = {nb, tiles, S};
      }
    }
  }
  return best;
}
// bytes of fp32 partial sums the plan writes (QKV always goes through them;
// the residual projections store [splits][Mp][N] row-major)
size_t plan_partial_bytes(int epi, const GemmPlan& p, int MT) {
  if (epi == EPI_QKV) return (size_t)MT * p.tiles * p.splits * p.nb * 16384;
  return p.splits > 1 ? (size_t)p.splits * MT * 256 * p.tiles * p.nb * 16 * 4 : 0;
}

}  // namespace

struct lopa_model {
  lopa_model_cfg cfg;
  int device = 0;
  int num_cu = 0;
  int n_qkv = 0;
  int blk_qkv = 0, blk_h = 0, blk_gu = 0, blk_lm = 0;  // packed 16-column blocks
  int nb_qkv = 0, nb_o = 0, nb_down = 0, nb_lm = 0;     // tile widths of the packed weights
  int tiles_lm = 0;                                     // LM-head column tiles
  int fp8 = 0;       // FP8 MLP (LOPA_PRECISION_FP8_MLP and LOPA_PRECISION_FP8)
  int fp8_qkv_lm = 0;  // FP8 QKV projection and LM head too (LOPA_PRECISION_FP8)
  int nb_down8 = 0;                                     // FP8 down-projection tile width
  int nb_o8 = 0;                                        // FP8 output-projection tile width
  std::vector<LayerPack> layers;
  uint16_t* embed = nullptr;
  uint16_t* lm = nullptr;   // bf16 LM head (when not FP8)
  uint8_t* lm8 = nullptr;   // FP8 LM head, K = round512(H), and its column scales
  float* sw_lm = nullptr;
  float* final_norm = nullptr;
  std::vector<void*> owned;
  ~lopa_model() {
    for (void* p : owned) (void)hipFree(p);
  }
};

struct lopa_kv {
  const lopa_model* m = nullptr;
  int max_len = 0, max_branches = 0, max_block = 0, mp_max = 0;
  int vld = 0, vlds = 0;        // positions per head region: max_len, max_block rounded up to 32
  uint16_t* cache = nullptr;    // [layers][2][Hkv][d * vld], KV tile layout (common.h)
  uint16_t* staging = nullptr;  // [max_branches][layers][2][Hkv][d * vlds]
  float* rope = nullptr;        // [max_len][d/2][2]
  float* x = nullptr;           // [mp_max][H]
  uint16_t* abuf = nullptr;     // packed [mp_max][H]
  uint16_t* fbuf = nullptr;     // packed [mp_max][round256(F)], padding columns zero
  // FP8 models: the FP8 operands of gate/up and down (padding columns zero)
  // and their per-row scales; a8_gu / sa_gu also carry the normed rows into
  // the QKV projection and the LM head of LOPA_PRECISION_FP8 models
  uint8_t* a8_gu = nullptr;     // packed [mp_max][round512(H)] E4M3
  uint8_t* a8_dn = nullptr;     // packed [mp_max][round512(F)] E4M3
  float* sa_gu = nullptr;
  float* sa_dn = nullptr;
  uint32_t* rowmax_dn = nullptr;  // per-row max |SwiGLU output| (float bits)
  uint16_t* qbuf = nullptr;     // [max_branches][Hq][max_block][d]
  float* partials = nullptr;
  int causal_blk = 0;           // lopa_kv_set_block_causal: 0 full attention in the block
  float* pm = nullptr;
  float* ps = nullptr;
  int32_t* pi = nullptr;
  int last_nb = -1, last_L = -1, last_P = -1;
  size_t part_bytes = 0;  // bytes of partials
  std::vector<void*> owned;
  // launch timing (lopa_kv_profile): events around launches of enabled kinds
  int prof_mask = 0;
  struct Ev {
    int kind;
    hipEvent_t a, b;
  };
  std::vector<Ev> ev_pool;
  size_t ev_used = 0;
  double prof_ms[LOPA_PROF_KINDS] = {};
  int64_t prof_n[LOPA_PROF_KINDS] = {};
  ~lopa_kv() {
    for (auto& e : ev_pool) {
      (void)hipEventDestroy(e.a);
      (void)hipEventDestroy(e.b);
    }
    for (void* p : owned) (void)hipFree(p);
  }
};

namespace {
// Record an event pair around one launch when its kind is enabled.
struct ProfScope {
  lopa_kv* kv;
  lopa_kv::Ev* ev = nullptr;
  hipStream_t s;
  ProfScope(lopa_kv* k, int kind, hipStream_t st) : kv(k), s(st) {
    if (!(kv->prof_mask & (1 << kind))) return;
    if (kv->ev_used == kv->ev_pool.size()) {
      lopa_kv::Ev e{kind, nullptr, nullptr};
      // timing only: no system-scope fence (its cache write-back would be
      // timed with the launch and slow the work after it)
      if (hipEventCreateWithFlags(&e.a, hipEventDisableSystemFence) != hipSuccess ||
          hipEventCreateWithFlags(&e.b, hipEventDisableSystemFence) != hipSuccess)
        return;
      kv->ev_pool.push_back(e);
    }
    ev = &kv->ev_pool[kv->ev_used++];
    ev->kind = kind;
    (void)hipEventRecord(ev->a, s);
  }
  ~ProfScope() {
    if (ev) (void)hipEventRecord(ev->b, s);
  }
};
// the plans of the five GEMMs of a verify forward with MT row tiles
struct StepPlans {
  GemmPlan qkv, o, gu, down, lm;
};
StepPlans step_plans(const lopa_model* m, int MT) {
  const lopa_model_cfg& c = m->cfg;
  StepPlans p;
  const int kch = m->fp8_qkv_lm ? round512(c.hidden) / 128 : c.hidden / 64;
  p.qkv = plan_gemm(EPI_QKV, m->blk_qkv, kch, MT, m->num_cu, m->nb_qkv);
  p.o = m->fp8_qkv_lm
            ? plan_gemm(EPI_RESID, m->blk_h, round512(c.heads * c.head_dim) / 128, MT, m->num_cu, m->nb_o8)
            : plan_gemm(EPI_RESID, m->blk_h, c.heads * c.head_dim / 64, MT, m->num_cu, m->nb_o);
  p.gu = plan_gemm(EPI_SWIGLU, m->blk_gu, c.hidden / 64, MT, m->num_cu, 10);
  p.down = m->fp8 ? plan_gemm(EPI_RESID, m->blk_h, round512(c.ffn) / 128, MT, m->num_cu, m->nb_down8)
                  : plan_gemm(EPI_RESID, m->blk_h, round256(c.ffn) / 64, MT, m->num_cu, m->nb_down);
  p.lm = plan_gemm(EPI_LMHEAD, m->blk_lm, kch, MT, m->num_cu, m->nb_lm);
  return p;
}
}  // namespace

extern "C" {

const char* lopa_strerror(int status) {
  switch (status) {
    case LOPA_OK: return "ok";
    case LOPA_EINVAL: return "invalid argument";
    case LOPA_ESHAPE: return "unsupported or over-capacity shape";
    case LOPA_ECAPACITY: return "KV cache capacity exceeded";
    case LOPA_EHIP: return "HIP runtime error";
    case LOPA_ENOMEM: return "device allocation failed";
  }
  return "unknown status";
}

const char* lopa_last_error(void) { return g_err.c_str(); }

static int check_cfg(const lopa_model_cfg* c) {
  if (!c) return fail(LOPA_EINVAL, "cfg is null");
  if (c->layers < 1 || c->hidden < 1 || c->heads < 1 || c->kv_heads < 1 || c->ffn < 1 ||
      c->vocab < 2)
    return fail(LOPA_EINVAL, "non-positive model dimension");
  if (c->mask_id < 0 || c->mask_id >= c->vocab)
    return fail(LOPA_EINVAL, "mask_id %d outside [0, %d)", c->mask_id, c->vocab);
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f) || !std::isfinite(c->rms_eps) ||
      !std::isfinite(c->rope_theta))
    return fail(LOPA_EINVAL, "rms_eps and rope_theta must be positive and finite");
  if (c->hidden % 256) return fail(LOPA_ESHAPE, "hidden %d is not a multiple of 256", c->hidden);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(LOPA_ESHAPE, "head_dim %d not in {64, 128}", c->head_dim);
  if (c->heads % c->kv_heads) return fail(LOPA_ESHAPE, "heads %% kv_heads != 0");
  if (c->heads * c->head_dim != c->hidden)
    return fail(LOPA_ESHAPE, "heads * head_dim != hidden");
  if (c->ffn % 64) return fail(LOPA_ESHAPE, "ffn %d is not a multiple of 64", c->ffn);
  return LOPA_OK;
}

int lopa_model_create(const lopa_model_cfg* cfg, const lopa_weight_ptrs* w, void* stream,
                      lopa_model** out) {
  return lopa_model_create_ex(cfg, w, LOPA_PRECISION_BF16, stream, out);
}

int lopa_model_create_ex(const lopa_model_cfg* cfg, const lopa_weight_ptrs* w, int32_t precision,
                         void* stream, lopa_model** out) {
  if (!out) return fail(LOPA_EINVAL, "out is null");
  if (precision != LOPA_PRECISION_BF16 && precision != LOPA_PRECISION_FP8_MLP &&
      precision != LOPA_PRECISION_FP8)
    return fail(LOPA_EINVAL, "unknown precision %d", precision);
  *out = nullptr;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!w || !w->embed || !w->layers || !w->final_norm || !w->lm_head)
    return fail(LOPA_EINVAL, "weight pointer is null");
  for (int l = 0; l < cfg->layers; ++l) {
    const lopa_layer_weights& lw = w->layers[l];
    if (!lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.w_gate || !lw.w_up || !lw.w_down ||
        !lw.ln1 || !lw.ln2)
      return fail(LOPA_EINVAL, "layer %d: weight pointer is null", l);
    if (cfg->qkv_bias && (!lw.bq || !lw.bk || !lw.bv))
      return fail(LOPA_EINVAL, "layer %d: qkv_bias set but a bias pointer is null", l);
  }
  hipStream_t s = (hipStream_t)stream;
  lopa_model* m = new lopa_model();
  m->cfg = *cfg;
  const lopa_model_cfg& c = *cfg;
  const int H = c.hidden, d = c.head_dim, F = c.ffn, V = c.vocab;
  m->n_qkv = (c.heads + 2 * c.kv_heads) * d;
  // blocks padded to whole tiles of every width a plan may pick (4, 8; 10 for
  // the gate / up pairs); padding blocks hold zero weights
  m->blk_qkv = round_up(m->n_qkv / 16, 8);
  m->blk_h = round_up(H / 16, 8);
  m->blk_gu = round_up(2 * F / 16, 10);
  auto bail = [&](int code) {
    delete m;
    return code;
  };
  if (hipGetDevice(&m->device) != hipSuccess ||
      hipDeviceGetAttribute(&m->num_cu, hipDeviceAttributeMultiprocessorCount, m->device) !=
          hipSuccess)
    return bail(fail(LOPA_EHIP, "no HIP device"));
  // LM head: 8- or 10-block tiles (whole tiles, no split: the epilogue reduces
  // each tile's softmax statistics), whichever gives fewer rounds of
  // workgroups x per-workgroup bytes (activation chunk + weights per k-chunk)
  {
    double best = 1e300;
    for (int nb : {8, 10}) {
      const int tiles = round_up((V + 15) / 16, nb) / nb;
      const double t = std::ceil((double)tiles / m->num_cu) * (32768.0 + nb * 2048.0);
      if (t < best) {
        best = t;
        m->nb_lm = nb;
      }
    }
  }
  m->blk_lm = round_up((V + 15) / 16, m->nb_lm);
  m->tiles_lm = m->blk_lm / m->nb_lm;
  // tile widths: those of the single-row-tile plans (up to 256 rows, the
  // common verify batch); other row counts re-plan the k-splits only
  m->nb_qkv = plan_gemm(EPI_QKV, m->blk_qkv, H / 64, 1, m->num_cu, 0).nb;
  m->nb_o = plan_gemm(EPI_RESID, m->blk_h, c.heads * d / 64, 1, m->num_cu, 0).nb;
  m->nb_down = plan_gemm(EPI_RESID, m->blk_h, round256(F) / 64, 1, m->num_cu, 0).nb;
  m->fp8 = precision == LOPA_PRECISION_FP8_MLP || precision == LOPA_PRECISION_FP8;
  m->fp8_qkv_lm = precision == LOPA_PRECISION_FP8;
  m->nb_down8 = plan_gemm(EPI_RESID, m->blk_h, round512(F) / 128, 1, m->num_cu, 0).nb;
  m->nb_o8 = plan_gemm(EPI_RESID, m->blk_h, round512(c.heads * d) / 128, 1, m->num_cu, 0).nb;
  auto alloc16 = [&](uint16_t** p, size_t elems) -> int {
    DevBuf b;
    int r = dalloc(b, elems * 2, m->owned);
    *p = (uint16_t*)b.p;
    return r;
  };
  auto allocf = [&](float** p, size_t elems) -> int {
    DevBuf b;
    int r = dalloc(b, elems * 4, m->owned);
    *p = (float*)b.p;
    return r;
  };
  const int FP = round256(F);  // down projection K, zero-padded
  const int KPH8 = round512(H), KPF8 = round512(F);  // FP8 MLP K, zero-padded
  // elements of a packed weight: blocks x K x 16
  auto wsize = [](int blocks, int K) { return (size_t)blocks * K * 16; };
  auto alloc8 = [&](uint8_t** p, size_t bytes) -> int {
    DevBuf b;
    int r = dalloc(b, bytes, m->owned);
    *p = (uint8_t*)b.p;
    return r;
  };
  // FP8: per source row scaling pairs (gate, up: F rows; down: H rows; q, k,
  // v: n_qkv rows; LM head: V rows)
  float *inv_g = nullptr, *sc_g = nullptr, *inv_u = nullptr, *sc_u = nullptr, *inv_d = nullptr,
        *sc_d = nullptr, *inv_q = nullptr, *sc_q = nullptr;
  if (m->fp8 && ((rc = allocf(&inv_g, F)) || (rc = allocf(&sc_g, F)) || (rc = allocf(&inv_u, F)) ||
                 (rc = allocf(&sc_u, F)) || (rc = allocf(&inv_d, H)) || (rc = allocf(&sc_d, H))))
    return bail(rc);
  if (m->fp8_qkv_lm &&
      ((rc = allocf(&inv_q, std::max(m->n_qkv, V))) || (rc = allocf(&sc_q, std::max(m->n_qkv, V)))))
    return bail(rc);
  const int nq = c.heads * d, nk = c.kv_heads * d;
  m->layers.resize(c.layers);
  for (int l = 0; l < c.layers; ++l) {
    const lopa_layer_weights& lw = w->layers[l];
    LayerPack& p = m->layers[l];
    p.gu = p.down = p.qkv = nullptr;
    if ((!m->fp8_qkv_lm && (rc = alloc16(&p.qkv, wsize(m->blk_qkv, H)))) ||
        (m->fp8_qkv_lm && (rc = alloc8(&p.qkv8, wsize(m->blk_qkv, KPH8)))) ||
        (m->fp8_qkv_lm && (rc = allocf(&p.sw_qkv, (size_t)m->blk_qkv * 16))) ||
        (!m->fp8_qkv_lm && (rc = alloc16(&p.o, wsize(m->blk_h, c.heads * d)))) ||
        (m->fp8_qkv_lm && (rc = alloc8(&p.o8, wsize(m->blk_h, round512(c.heads * d))))) ||
        (m->fp8_qkv_lm && (rc = allocf(&p.sw_o, (size_t)m->blk_h * 16))) ||
        (!m->fp8 && (rc = alloc16(&p.gu, wsize(m->blk_gu, H)))) ||
        (!m->fp8 && (rc = alloc16(&p.down, wsize(m->blk_h, FP)))) ||
        (m->fp8 && (rc = alloc8(&p.gu8, wsize(m->blk_gu, KPH8)))) ||
        (m->fp8 && (rc = alloc8(&p.down8, wsize(m->blk_h, KPF8)))) ||
        (m->fp8 && (rc = allocf(&p.sw_gu, (size_t)m->blk_gu * 16))) ||
        (m->fp8 && (rc = allocf(&p.sw_down, (size_t)m->blk_h * 16))) ||
        (rc = allocf(&p.ln1, H)) || (rc = allocf(&p.ln2, H)))
      return bail(rc);
    p.bias = nullptr;
    if (c.qkv_bias && (rc = allocf(&p.bias, m->n_qkv))) return bail(rc);
    const uint16_t* wq = (const uint16_t*)lw.wq;
    const uint16_t* wk = (const uint16_t*)lw.wk;
    const uint16_t* wv = (const uint16_t*)lw.wv;
    hipError_t e;
    if ((!m->fp8_qkv_lm &&
         (e = launch_repack(wq, nq, wk, nk, wv, nk, H, H, m->blk_qkv, m->nb_qkv, 0, p.qkv, s)) !=
             hipSuccess) ||
        (m->fp8_qkv_lm &&
         ((e = launch_rowscale(wq, nq, H, inv_q, sc_q, s)) != hipSuccess ||
          (e = launch_rowscale(wk, nk, H, inv_q + nq, sc_q + nq, s)) != hipSuccess ||
          (e = launch_rowscale(wv, nk, H, inv_q + nq + nk, sc_q + nq + nk, s)) != hipSuccess ||
          (e = launch_repack8(wq, inv_q, sc_q, nq, wk, inv_q + nq, sc_q + nq, nk, wv,
                              inv_q + nq + nk, sc_q + nq + nk, nk, H, KPH8, m->blk_qkv,
                              m->nb_qkv, 0, p.qkv8, p.sw_qkv, s)) != hipSuccess)) ||
        (!m->fp8_qkv_lm &&
         (e = launch_repack((const uint16_t*)lw.wo, H, nullptr, 0, nullptr, 0, c.heads * d,
                            c.heads * d, m->blk_h, m->nb_o, 0, p.o, s)) != hipSuccess) ||
        (m->fp8_qkv_lm &&  // the row-scale buffers are free again: the QKV repack ran before
         ((e = launch_rowscale((const uint16_t*)lw.wo, H, c.heads * d, inv_q, sc_q, s)) !=
              hipSuccess ||
          (e = launch_repack8((const uint16_t*)lw.wo, inv_q, sc_q, H, nullptr, nullptr, nullptr, 0,
                              nullptr, nullptr, nullptr, 0, c.heads * d, round512(c.heads * d),
                              m->blk_h, m->nb_o8, 0, p.o8, p.sw_o, s)) != hipSuccess)) ||
        (!m->fp8 &&
         (e = launch_repack((const uint16_t*)lw.w_gate, F, (const uint16_t*)lw.w_up, F, nullptr,
                            0, H, H, m->blk_gu, 10, 1, p.gu, s)) != hipSuccess) ||
        (!m->fp8 &&
         (e = launch_repack((const uint16_t*)lw.w_down, H, nullptr, 0, nullptr, 0, F, FP,
                            m->blk_h, m->nb_down, 0, p.down, s)) != hipSuccess) ||
        (m->fp8 &&
         ((e = launch_rowscale((const uint16_t*)lw.w_gate, F, H, inv_g, sc_g, s)) != hipSuccess ||
          (e = launch_rowscale((const uint16_t*)lw.w_up, F, H, inv_u, sc_u, s)) != hipSuccess ||
          (e = launch_rowscale((const uint16_t*)lw.w_down, H, F, inv_d, sc_d, s)) != hipSuccess ||
          (e = launch_repack8((const uint16_t*)lw.w_gate, inv_g, sc_g, F,
                              (const uint16_t*)lw.w_up, inv_u, sc_u, F, nullptr, nullptr, nullptr,
                              0, H, KPH8, m->blk_gu, 10, 1, p.gu8, p.sw_gu, s)) != hipSuccess ||
          (e = launch_repack8((const uint16_t*)lw.w_down, inv_d, sc_d, H, nullptr, nullptr,
                              nullptr, 0, nullptr, nullptr, nullptr, 0, F, KPF8, m->blk_h,
                              m->nb_down8, 0, p.down8, p.sw_down, s)) != hipSuccess)) ||
        (e = launch_bf16_to_f32((const uint16_t*)lw.ln1, p.ln1, H, s)) != hipSuccess ||
        (e = launch_bf16_to_f32((const uint16_t*)lw.ln2, p.ln2, H, s)) != hipSuccess)
      return bail(fail(LOPA_EHIP, "layer %d repack: %s", l, hipGetErrorString(e)));
    if (p.bias) {
      if ((e = launch_bf16_to_f32((const uint16_t*)lw.bq, p.bias, c.heads * d, s)) ||
          (e = launch_bf16_to_f32((const uint16_t*)lw.bk, p.bias + c.heads * d, c.kv_heads * d,
                                  s)) ||
          (e = launch_bf16_to_f32((const uint16_t*)lw.bv,
                                  p.bias + (c.heads + c.kv_heads) * d, c.kv_heads * d, s)))
        return bail(fail(LOPA_EHIP, "layer %d bias: %s", l, hipGetErrorString(e)));
    }
  }
  if ((rc = alloc16(&m->embed, (size_t)V * H)) ||
      (!m->fp8_qkv_lm && (rc = alloc16(&m->lm, wsize(m->blk_lm, H)))) ||
      (m->fp8_qkv_lm && (rc = alloc8(&m->lm8, wsize(m->blk_lm, KPH8)))) ||
      (m->fp8_qkv_lm && (rc = allocf(&m->sw_lm, (size_t)m->blk_lm * 16))) ||
      (rc = allocf(&m->final_norm, H)))
    return bail(rc);
  hipError_t e;
  const uint16_t* lmw = (const uint16_t*)w->lm_head;
  if ((e = hipMemcpyAsync(m->embed, w->embed, (size_t)V * H * 2, hipMemcpyDeviceToDevice, s)) ||
      (!m->fp8_qkv_lm && (e = launch_repack(lmw, V, nullptr, 0, nullptr, 0, H, H, m->blk_lm,
                                            m->nb_lm, 0, m->lm, s))) ||
      (m->fp8_qkv_lm &&
       ((e = launch_rowscale(lmw, V, H, inv_q, sc_q, s)) ||
        (e = launch_repack8(lmw, inv_q, sc_q, V, nullptr, nullptr, nullptr, 0, nullptr, nullptr,
                            nullptr, 0, H, KPH8, m->blk_lm, m->nb_lm, 0, m->lm8, m->sw_lm, s)))) ||
      (e = launch_bf16_to_f32((const uint16_t*)w->final_norm, m->final_norm, H, s)) ||
      (e = hipStreamSynchronize(s)))
    return bail(fail(LOPA_EHIP, "model create: %s", hipGetErrorString(e)));
  *out = m;
  return LOPA_OK;
}

void lopa_model_destroy(lopa_model* m) { delete m; }

int lopa_kv_create(const lopa_model* m, int32_t max_len, int32_t max_branches, int32_t max_block,
                   lopa_kv** out) {
  if (!out) return fail(LOPA_EINVAL, "out is null");
  *out = nullptr;
  if (!m) return fail(LOPA_EINVAL, "model is null");
  if (max_len < 1 || max_branches < 1 || max_block < 1)
    return fail(LOPA_EINVAL, "max_len, max_branches and max_block must be positive");
  if (max_block > LOPA_MAX_BLOCK)
    return fail(LOPA_ESHAPE, "max_block %d > %d", max_block, LOPA_MAX_BLOCK);
  if ((int64_t)max_branches * max_block > LOPA_MAX_ROWS)
    return fail(LOPA_ESHAPE, "max_branches * max_block > %d", LOPA_MAX_ROWS);
  const lopa_model_cfg& c = m->cfg;
  lopa_kv* kv = new lopa_kv();
  kv->m = m;
  kv->max_len = max_len;
  kv->max_branches = max_branches;
  kv->max_block = max_block;
  kv->mp_max = padded_rows(max_branches * max_block);
  const int H = c.hidden, F = c.ffn, d = c.head_dim, Hkv = c.kv_heads;
  auto bail = [&](int code) {
    delete kv;
    return code;
  };
  DevBuf b;
  int rc;
  kv->vld = round_up(max_len, 32);  // whole KV tiles (32 positions)
  kv->vlds = round_up(max_block, 32);
  const size_t cache_e = (size_t)c.layers * 2 * Hkv * d * kv->vld;
  const size_t stag_e = (size_t)max_branches * c.layers * 2 * Hkv * d * kv->vlds;
  size_t part_b = 16;
  for (int MT = 1; MT <= kv->mp_max / 256; ++MT) {
    const StepPlans p = step_plans(m, MT);
    part_b = std::max({part_b, plan_partial_bytes(EPI_QKV, p.qkv, MT),
                       plan_partial_bytes(EPI_RESID, p.o, MT),
                       plan_partial_bytes(EPI_RESID, p.down, MT)});
  }
  // the attention's scratch (between the QKV fix-up and the output projection
  // the partial sums are free): its largest need over the branch counts
  for (int nb = 1; nb <= max_branches; ++nb)
    part_b = std::max(part_b, attention_scratch_bytes(nb, std::min(max_block, 32), c.heads,
                                                      c.kv_heads, d));
  kv->part_bytes = part_b;
  const size_t rows = (size_t)kv->mp_max;
  const int FP = round256(F);
#define KV_ALLOC(field, type, bytes)                  \
  if ((rc = dalloc(b, (bytes), kv->owned))) return bail(rc); \
  kv->field = (type)b.p;
  KV_ALLOC(cache, uint16_t*, cache_e * 2);
  KV_ALLOC(staging, uint16_t*, stag_e * 2);
  KV_ALLOC(rope, float*, (size_t)max_len * (d / 2) * 2 * 4);
  KV_ALLOC(x, float*, rows * H * 4);
  KV_ALLOC(abuf, uint16_t*, rows * H * 2);
  KV_ALLOC(fbuf, uint16_t*, rows * FP * 2);
  if (m->fp8) {
    KV_ALLOC(a8_gu, uint8_t*, rows * round512(H));
    KV_ALLOC(a8_dn, uint8_t*, rows * round512(F));
    KV_ALLOC(sa_gu, float*, rows * 4);
    KV_ALLOC(sa_dn, float*, rows * 4);
    KV_ALLOC(rowmax_dn, uint32_t*, rows * 4);
  }
  KV_ALLOC(qbuf, uint16_t*, (size_t)max_branches * c.heads * max_block * d * 2);
  KV_ALLOC(partials, float*, part_b);
  KV_ALLOC(pm, float*, rows * m->tiles_lm * 4);
  KV_ALLOC(ps, float*, rows * m->tiles_lm * 4);
  KV_ALLOC(pi, int32_t*, rows * m->tiles_lm * 4);
#undef KV_ALLOC
  // RoPE table in double precision, stored as fp32 (cos, sin) pairs.
  std::vector<float> tab((size_t)max_len * (d / 2) * 2);
  for (int p = 0; p < max_len; ++p)
    for (int j = 0; j < d / 2; ++j) {
      const double inv = std::pow((double)c.rope_theta, -2.0 * j / d);
      const double ang = (double)p * inv;
      tab[((size_t)p * (d / 2) + j) * 2] = (float)std::cos(ang);
      tab[((size_t)p * (d / 2) + j) * 2 + 1] = (float)std::sin(ang);
    }
  hipError_t e;
  if ((e = hipMemcpy(kv->rope, tab.data(), tab.size() * 4, hipMemcpyHostToDevice)) ||
      (e = hipMemset(kv->cache, 0, cache_e * 2)) || (e = hipMemset(kv->staging, 0, stag_e * 2)) ||
      (e = hipMemset(kv->abuf, 0, rows * H * 2)) || (e = hipMemset(kv->fbuf, 0, rows * FP * 2)) ||
      (m->fp8 && ((e = hipMemset(kv->a8_gu, 0, rows * round512(H))) ||
                  (e = hipMemset(kv->a8_dn, 0, rows * round512(F))) ||
                  (e = hipMemset(kv->sa_gu, 0, rows * 4)) ||
                  (e = hipMemset(kv->sa_dn, 0, rows * 4)))) ||
      (e = hipDeviceSynchronize()))
    return bail(fail(LOPA_EHIP, "kv create: %s", hipGetErrorString(e)));
  *out = kv;
  return LOPA_OK;
}

void lopa_kv_destroy(lopa_kv* kv) { delete kv; }

int lopa_build_branches_window(const int32_t* tokens, const float* conf, const int32_t* pred,
                               int32_t L, int32_t n_eligible, int32_t mask_id, float tau,
                               int32_t k, int32_t* branch_tokens, int32_t* fill_pos,
                               uint8_t* valid, int32_t* n_valid, void* stream) {
  if (!tokens || !conf || !pred || !branch_tokens || !fill_pos || !valid || !n_valid)
    return fail(LOPA_EINVAL, "null pointer argument");
  if (k < 0) return fail(LOPA_EINVAL, "k = %d < 0", k);
  if (!(tau >= 0.f && tau <= 1.f)) return fail(LOPA_EINVAL, "tau outside [0, 1]");
  if (mask_id < 0) return fail(LOPA_EINVAL, "mask_id < 0");
  if (L < 1 || L > LOPA_MAX_BLOCK) return fail(LOPA_ESHAPE, "L = %d outside [1, %d]", L, LOPA_MAX_BLOCK);
  if (n_eligible < 1 || n_eligible > L)
    return fail(LOPA_EINVAL, "n_eligible = %d outside [1, L = %d]", n_eligible, L);
  if (k + 1 > LOPA_MAX_ROWS) return fail(LOPA_ESHAPE, "k = %d too large", k);
  HIP_TRY(launch_build_branches(tokens, conf, pred, L, n_eligible, mask_id, tau, k, branch_tokens,
                                fill_pos, valid, n_valid, (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_build_branches(const int32_t* tokens, const float* conf, const int32_t* pred,
                        int32_t L, int32_t mask_id, float tau, int32_t k, int32_t* branch_tokens,
                        int32_t* fill_pos, uint8_t* valid, int32_t* n_valid, void* stream) {
  return lopa_build_branches_window(tokens, conf, pred, L, L < 1 ? 1 : L, mask_id, tau, k,
                                    branch_tokens, fill_pos, valid, n_valid, stream);
}

// The verify forward; with stop_layer >= 0 it stops after that many layers and
// copies the fp32 residual stream to x_out instead of producing conf / pred.
static int verify_impl(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                       const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                       int32_t* pred, void* stream, int stop_layer, float* x_out,
                       const VerifyWs& ws) {
  const lopa_model_cfg& c = m->cfg;
  hipStream_t s = (hipStream_t)stream;
  const int M = n_branches * L;
  const int Mp = padded_rows(M);
  const int H = c.hidden, F = c.ffn, d = c.head_dim;
  const int MT = Mp / 256;
  const StepPlans plan = step_plans(m, MT);

  GemmArgs g{};
  g.M = M;
  g.Mp = Mp;
  g.mtiles = MT;
  g.partials = ws.partials;
  auto gemm = [&](int epi, const uint16_t* A, const uint16_t* W, int N, int K,
                  const GemmPlan& p) {
    g.A = A;
    g.W = W;
    g.N = N;
    g.KC = K / 64;
    g.rot = epi == EPI_SWIGLU || epi == EPI_RESID;
    g.f8 = 0;
    g.sa = g.sw = nullptr;
    g.nb = p.nb;
    g.tiles = p.tiles;
    g.splits = p.splits;
    g.gcols = p.tiles * p.splits;
    return launch_gemm(epi, g, s);
  };
  // FP8 operands: A, W E4M3 with K = KP (a multiple of 512), row / column scales
  auto gemm8 = [&](int epi, const uint8_t* A, const uint8_t* W, int N, int KP, const float* sa,
                   const float* sw, const GemmPlan& pl) {
    g.A = (const uint16_t*)A;
    g.W = (const uint16_t*)W;
    g.N = N;
    g.KC = KP / 128;
    g.rot = epi == EPI_SWIGLU || epi == EPI_RESID;
    g.f8 = 1;
    g.sa = sa;
    g.sw = sw;
    g.rowmax = ws.rowmax_dn;
    g.nb = pl.nb;
    g.tiles = pl.tiles;
    g.splits = pl.splits;
    g.gcols = pl.tiles * pl.splits;
    return launch_gemm(epi, g, s);
  };
  const bool f8x = m->fp8_qkv_lm;  // the normed rows go to the QKV / LM head in E4M3

  { ProfScope ps_(kv, LOPA_PROF_NORM, s);
    if (f8x)
      HIP_TRY(launch_embed_norm8(branch_tokens, m->embed, c.vocab, m->layers[0].ln1, c.rms_eps, M,
                                 Mp, H, ws.x, ws.a8_gu, ws.sa_gu, ws.rowmax_dn, s));
    else
      HIP_TRY(launch_embed_norm(branch_tokens, m->embed, c.vocab, m->layers[0].ln1, c.rms_eps, M,
                                Mp, H, ws.x, ws.abuf, s)); }
  AttnArgs at{};
  at.q = ws.qbuf;
  at.staging = kv->staging;
  at.out = ws.abuf;
  at.nb = n_branches;
  at.L = L;
  at.P = prefix_len;
  at.Hq = c.heads;
  at.Hkv = c.kv_heads;
  at.d = d;
  at.vld = kv->vld;
  at.layers = c.layers;
  at.vlds = kv->vlds;
  at.Mp = Mp;
  at.scale = 1.0f / std::sqrt((float)d);
  // a block of one sub-block (or less) needs no mask
  at.cblk = kv->causal_blk && L > kv->causal_blk ? kv->causal_blk : 0;
  at.scratch = ws.partials;
  at.scratch_bytes = ws.partials_bytes;
  // FP8 output projection: the attention output's row maxima, in the buffer
  // the norm ahead of each layer's QKV projection zeroes (the gate/up GEMM's
  // row maxima use it again after the second norm zeroes it)
  at.rowmax = f8x ? ws.rowmax_dn : nullptr;
  const int n_layers = stop_layer >= 0 ? std::min(stop_layer, c.layers) : c.layers;
  for (int l = 0; l < n_layers; ++l) {
    const LayerPack& p = m->layers[l];
    g.bias = p.bias;
    g.rope = kv->rope;
    g.q_out = ws.qbuf;
    g.staging = kv->staging;
    g.layer = l;
    g.layers = c.layers;
    g.Hq = c.heads;
    g.Hkv = c.kv_heads;
    g.d = d;
    g.L = L;
    g.vlds = kv->vlds;
    g.P = prefix_len;
    { ProfScope ps_(kv, LOPA_PROF_QKV, s);
      if (f8x)
        HIP_TRY(gemm8(EPI_QKV, ws.a8_gu, p.qkv8, m->n_qkv, round512(H), ws.sa_gu, p.sw_qkv,
                      plan.qkv));
      else
        HIP_TRY(gemm(EPI_QKV, ws.abuf, p.qkv, m->n_qkv, H, plan.qkv)); }
    at.layer = l;
    at.kcache = kv->cache + ((size_t)l * 2 + 0) * c.kv_heads * d * kv->vld;
    at.vcache = kv->cache + ((size_t)l * 2 + 1) * c.kv_heads * d * kv->vld;
    { ProfScope ps_(kv, LOPA_PROF_ATTN, s);
      HIP_TRY(launch_attention(at, s)); }
    g.x = ws.x;
    if (f8x) {
      // FP8 output projection: the attention output (bf16) to E4M3 with a
      // scale per row over all heads (the row maxima the attention kernels
      // merged), in the operand buffer of the QKV projection, which has read
      // it by now
      { ProfScope ps_(kv, LOPA_PROF_NORM, s);
        HIP_TRY(launch_quant_rows8(ws.abuf, c.heads * d, M, Mp, ws.rowmax_dn, ws.a8_gu, ws.sa_gu,
                                   s)); }
      { ProfScope ps_(kv, LOPA_PROF_OPROJ, s);
        HIP_TRY(gemm8(EPI_RESID, ws.a8_gu, p.o8, H, round512(c.heads * d), ws.sa_gu, p.sw_o,
                      plan.o)); }
    } else {
      ProfScope ps_(kv, LOPA_PROF_OPROJ, s);
      HIP_TRY(gemm(EPI_RESID, ws.abuf, p.o, H, c.heads * d, plan.o));
    }
    g.a_out = ws.fbuf;
    if (m->fp8) {
      // FP8 MLP: the normed rows straight to E4M3 with their scales, gate/up,
      // the SwiGLU output (bf16) requantised per row, down
      { ProfScope ps_(kv, LOPA_PROF_NORM, s);
        HIP_TRY(launch_resnorm8(ws.partials, plan.o.splits > 1 ? plan.o.splits : 0, p.ln2,
                                c.rms_eps, M, Mp, H, ws.x, ws.a8_gu, ws.sa_gu, ws.rowmax_dn,
                                s)); }
      { ProfScope ps_(kv, LOPA_PROF_GATEUP, s);
        HIP_TRY(gemm8(EPI_SWIGLU, ws.a8_gu, p.gu8, 2 * F, round512(H), ws.sa_gu, p.sw_gu,
                      plan.gu)); }
      { ProfScope ps_(kv, LOPA_PROF_NORM, s);
        HIP_TRY(launch_quant_rows8(ws.fbuf, F, M, Mp, ws.rowmax_dn, ws.a8_dn, ws.sa_dn, s)); }
      { ProfScope ps_(kv, LOPA_PROF_DOWN, s);
        HIP_TRY(gemm8(EPI_RESID, ws.a8_dn, p.down8, H, round512(F), ws.sa_dn, p.sw_down,
                      plan.down)); }
    } else {
      { ProfScope ps_(kv, LOPA_PROF_NORM, s);
        HIP_TRY(launch_resnorm(ws.partials, plan.o.splits > 1 ? plan.o.splits : 0, p.ln2,
                               c.rms_eps, M, Mp, H, ws.x, ws.abuf, s)); }
      { ProfScope ps_(kv, LOPA_PROF_GATEUP, s);
        HIP_TRY(gemm(EPI_SWIGLU, ws.abuf, p.gu, 2 * F, H, plan.gu)); }
      { ProfScope ps_(kv, LOPA_PROF_DOWN, s);
        HIP_TRY(gemm(EPI_RESID, ws.fbuf, p.down, H, round256(F), plan.down)); }
    }
    const float* next_w = (l + 1 < c.layers) ? m->layers[l + 1].ln1 : m->final_norm;
    const int dsplits = plan.down.splits > 1 ? plan.down.splits : 0;
    { ProfScope ps_(kv, LOPA_PROF_NORM, s);
      if (f8x)  // also zeroes the row maxima for the next layer's attention output
        HIP_TRY(launch_resnorm8(ws.partials, dsplits, next_w, c.rms_eps, M, Mp, H, ws.x,
                                ws.a8_gu, ws.sa_gu, ws.rowmax_dn, s));
      else
        HIP_TRY(launch_resnorm(ws.partials, dsplits, next_w, c.rms_eps, M, Mp, H, ws.x,
                               ws.abuf, s)); }
  }
  if (stop_layer >= 0) {
    HIP_TRY(hipMemcpyAsync(x_out, ws.x, (size_t)M * H * 4, hipMemcpyDeviceToDevice, s));
    return LOPA_OK;
  }
  g.pm = ws.pm;
  g.ps = ws.ps;
  g.pi = ws.pi;
  g.vocab = c.vocab;
  g.mask_id = c.mask_id;
  { ProfScope ps_(kv, LOPA_PROF_LMHEAD, s);
    if (f8x)
      HIP_TRY(gemm8(EPI_LMHEAD, ws.a8_gu, m->lm8, c.vocab, round512(H), ws.sa_gu, m->sw_lm,
                    plan.lm));
    else
      HIP_TRY(gemm(EPI_LMHEAD, ws.abuf, m->lm, c.vocab, H, plan.lm)); }
  { ProfScope ps_(kv, LOPA_PROF_MERGE, s);
    HIP_TRY(launch_lm_merge(ws.pm, ws.ps, ws.pi, M, m->tiles_lm, conf, pred, s)); }
  kv->last_nb = n_branches;
  kv->last_L = L;
  kv->last_P = prefix_len;
  return LOPA_OK;
}

static int check_verify(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                        const int32_t* branch_tokens, int32_t n_branches, int32_t L) {
  if (!m || !kv || !branch_tokens) return fail(LOPA_EINVAL, "null pointer argument");
  if (kv->m != m) return fail(LOPA_EINVAL, "kv was created for another model");
  if (n_branches < 1 || L < 1) return fail(LOPA_ESHAPE, "n_branches and L must be >= 1");
  if (n_branches > kv->max_branches || L > kv->max_block)
    return fail(LOPA_ESHAPE, "n_branches %d / L %d exceed kv capacity %d / %d", n_branches, L,
                kv->max_branches, kv->max_block);
  if (prefix_len < 0) return fail(LOPA_EINVAL, "prefix_len < 0");
  if ((int64_t)prefix_len + L > kv->max_len)
    return fail(LOPA_ECAPACITY, "prefix_len %d + L %d > max_len %d", prefix_len, L, kv->max_len);
  if (kv->causal_blk && L > kv->causal_blk && L % kv->causal_blk)
    return fail(LOPA_ESHAPE, "L %d is not a multiple of the block-causal sub-block %d", L,
                kv->causal_blk);
  return LOPA_OK;
}

// the working buffers the KV handle owns (allocated by lopa_kv_create)
static VerifyWs kv_ws(const lopa_kv* kv) {
  VerifyWs w;
  w.x = kv->x;
  w.abuf = kv->abuf;
  w.fbuf = kv->fbuf;
  w.qbuf = kv->qbuf;
  w.partials = kv->partials;
  w.partials_bytes = kv->part_bytes;
  w.pm = kv->pm;
  w.ps = kv->ps;
  w.pi = kv->pi;
  w.a8_gu = kv->a8_gu;
  w.a8_dn = kv->a8_dn;
  w.sa_gu = kv->sa_gu;
  w.sa_dn = kv->sa_dn;
  w.rowmax_dn = kv->rowmax_dn;
  return w;
}

int lopa_verify_forward(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                        const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                        int32_t* pred, void* stream) {
  int rc = verify_check(m, kv, prefix_len, branch_tokens, n_branches, L, conf, pred);
  if (rc) return rc;
  return verify_impl(m, kv, prefix_len, branch_tokens, n_branches, L, conf, pred, stream, -1,
                     nullptr, kv_ws(kv));
}

int lopa_debug_hidden(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                      const int32_t* branch_tokens, int32_t n_branches, int32_t L,
                      int32_t n_layers, float* x_out, void* stream) {
  if (!x_out) return fail(LOPA_EINVAL, "null pointer argument");
  int rc = check_verify(m, kv, prefix_len, branch_tokens, n_branches, L);
  if (rc) return rc;
  if (n_layers < 0 || n_layers > m->cfg.layers) return fail(LOPA_EINVAL, "n_layers out of range");
  return verify_impl(m, kv, prefix_len, branch_tokens, n_branches, L, nullptr, nullptr, stream,
                     n_layers, x_out, kv_ws(kv));
}

int lopa_branch_confidence_select_metric(const int32_t* branch_tokens, const float* conf,
                                         const int32_t* pred, const uint8_t* valid,
                                         int32_t n_branches, int32_t L, int32_t mask_id,
                                         int32_t metric, int32_t window, float eta, float* scores,
                                         int32_t* winner, int32_t* next_tokens, float* next_conf,
                                         int32_t* next_pred, int32_t* next_unfilled,
                                         void* stream) {
  if (!branch_tokens || !conf || !pred || !valid || !scores || !winner || !next_tokens ||
      !next_conf || !next_pred || !next_unfilled)
    return fail(LOPA_EINVAL, "null pointer argument");
  if (n_branches < 1 || n_branches > 1024) return fail(LOPA_ESHAPE, "n_branches %d outside [1, 1024]", n_branches);
  if (L < 1 || L > LOPA_MAX_BLOCK) return fail(LOPA_ESHAPE, "L = %d outside [1, %d]", L, LOPA_MAX_BLOCK);
  if (mask_id < 0) return fail(LOPA_EINVAL, "mask_id < 0");
  if (metric < LOPA_METRIC_MEAN || metric > LOPA_METRIC_LOWEST_SEGMENT)
    return fail(LOPA_EINVAL, "unknown branch confidence metric %d", metric);
  if (metric == LOPA_METRIC_WINDOW_MIN && window < 1) return fail(LOPA_EINVAL, "window %d < 1", window);
  if (metric == LOPA_METRIC_LOWEST_SEGMENT && !(eta > 0.f && eta <= 1.f))
    return fail(LOPA_EINVAL, "eta outside (0, 1]");
  HIP_TRY(launch_select(branch_tokens, conf, pred, valid, n_branches, L, mask_id, metric, window,
                        eta, scores, winner, next_tokens, next_conf, next_pred, next_unfilled,
                        (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_branch_confidence_select(const int32_t* branch_tokens, const float* conf,
                                  const int32_t* pred, const uint8_t* valid, int32_t n_branches,
                                  int32_t L, int32_t mask_id, float* scores, int32_t* winner,
                                  int32_t* next_tokens, float* next_conf, int32_t* next_pred,
                                  int32_t* next_unfilled, void* stream) {
  return lopa_branch_confidence_select_metric(branch_tokens, conf, pred, valid, n_branches, L,
                                              mask_id, LOPA_METRIC_MEAN, 1, 1.f, scores, winner,
                                              next_tokens, next_conf, next_pred, next_unfilled,
                                              stream);
}

int lopa_commit_kv_rows(lopa_kv* kv, const int32_t* winner, int32_t prefix_len, int32_t L,
                        int32_t n_rows, int32_t* append_offset, void* stream) {
  if (!kv || !winner || !append_offset) return fail(LOPA_EINVAL, "null pointer argument");
  if (kv->last_nb < 0) return fail(LOPA_EINVAL, "no verify forward has staged K/V yet");
  if (prefix_len != kv->last_P || L != kv->last_L)
    return fail(LOPA_EINVAL, "prefix_len/L (%d, %d) differ from the last verify forward (%d, %d)",
                prefix_len, L, kv->last_P, kv->last_L);
  if (n_rows < 1 || n_rows > L) return fail(LOPA_EINVAL, "n_rows = %d outside [1, L = %d]", n_rows, L);
  if ((int64_t)prefix_len + n_rows > kv->max_len) return fail(LOPA_ECAPACITY, "commit beyond max_len");
  const lopa_model_cfg& c = kv->m->cfg;
  HIP_TRY(launch_commit(kv->staging, kv->cache, winner, kv->last_nb, c.layers, c.kv_heads,
                        kv->vlds, kv->vld, c.head_dim, prefix_len, n_rows, append_offset,
                        (hipStream_t)stream));
  return LOPA_OK;
}

// smallest filled count n of an L-position block with n / L >= tau (the
// gate's fraction in double), L + 1 if none
static int32_t gate_count(double tau, int32_t L) {
  for (int32_t n = 0; n <= L; ++n)
    if ((double)n / (double)L >= tau) return n;
  return L + 1;
}

int lopa_window_init(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred, int32_t L,
                     int32_t w_max, int32_t n_blocks, int32_t prefix_len, int32_t mask_id,
                     double tau_add, double tau_act, void* stream) {
  if (!win || !tokens || !conf || !pred) return fail(LOPA_EINVAL, "null pointer argument");
  if (L < 1 || w_max < 1 || w_max > LOPA_WINDOW_MAX_BLOCKS || (int64_t)w_max * L > LOPA_MAX_BLOCK)
    return fail(LOPA_ESHAPE, "window of %d blocks of %d positions (at most %d blocks, %d positions)",
                w_max, L, LOPA_WINDOW_MAX_BLOCKS, LOPA_MAX_BLOCK);
  if (n_blocks < 1 || prefix_len < 0) return fail(LOPA_EINVAL, "n_blocks %d, prefix_len %d", n_blocks, prefix_len);
  if (!(tau_add >= 0.0 && tau_add <= 1.0) || !(tau_act >= 0.0 && tau_act <= 1.0))
    return fail(LOPA_EINVAL, "tau_add %g / tau_act %g outside [0, 1]", tau_add, tau_act);
  const hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_window_init(win, L, w_max, n_blocks, prefix_len, mask_id, gate_count(tau_add, L),
                             gate_count(tau_act, L), s));
  HIP_TRY(launch_window_update(win, tokens, conf, pred, nullptr, s));
  return LOPA_OK;
}

int lopa_window_update(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred,
                       int32_t* out_tokens, void* stream) {
  if (!win || !tokens || !conf || !pred || !out_tokens) return fail(LOPA_EINVAL, "null pointer argument");
  HIP_TRY(launch_window_update(win, tokens, conf, pred, out_tokens, (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_window_commit(lopa_kv* kv, const int32_t* winner, lopa_window* win, void* stream) {
  if (!kv || !winner || !win) return fail(LOPA_EINVAL, "null pointer argument");
  if (kv->last_nb < 0) return fail(LOPA_EINVAL, "no verify forward has staged K/V yet");
  const lopa_model_cfg& c = kv->m->cfg;
  HIP_TRY(launch_window_commit(kv->staging, kv->cache, winner, win, kv->last_nb, kv->last_L,
                               kv->max_len, c.layers, c.kv_heads, kv->vlds, kv->vld, c.head_dim,
                               (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_commit_kv(lopa_kv* kv, const int32_t* winner, int32_t prefix_len, int32_t L,
                   int32_t* append_offset, void* stream) {
  if (!kv || !winner || !append_offset) return fail(LOPA_EINVAL, "null pointer argument");
  if (kv->last_nb < 0) return fail(LOPA_EINVAL, "no verify forward has staged K/V yet");
  if (prefix_len != kv->last_P || L != kv->last_L)
    return fail(LOPA_EINVAL, "prefix_len/L (%d, %d) differ from the last verify forward (%d, %d)",
                prefix_len, L, kv->last_P, kv->last_L);
  if ((int64_t)prefix_len + L > kv->max_len) return fail(LOPA_ECAPACITY, "commit beyond max_len");
  const lopa_model_cfg& c = kv->m->cfg;
  HIP_TRY(launch_commit(kv->staging, kv->cache, winner, kv->last_nb, c.layers, c.kv_heads,
                        kv->vlds, kv->vld, c.head_dim, prefix_len, L, append_offset,
                        (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_kv_read(const lopa_kv* kv, int32_t layer, int32_t start, int32_t len, void* k_dst,
                 void* v_dst, void* stream) {
  if (!kv || !k_dst || !v_dst) return fail(LOPA_EINVAL, "null pointer argument");
  const lopa_model_cfg& c = kv->m->cfg;
  if (layer < 0 || layer >= c.layers || start < 0 || len < 1 || (int64_t)start + len > kv->max_len)
    return fail(LOPA_EINVAL, "layer/start/len out of range");
  const int d = c.head_dim, Hkv = c.kv_heads;
  uint16_t* ck = kv->cache + ((size_t)layer * 2 + 0) * Hkv * d * kv->vld;
  uint16_t* cv = kv->cache + ((size_t)layer * 2 + 1) * Hkv * d * kv->vld;
  HIP_TRY(launch_kv_rows(ck, cv, (int64_t)d * kv->vld, kv->vld, Hkv, d, start, len,
                         (uint16_t*)k_dst, (uint16_t*)v_dst, 0, (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_kv_write(lopa_kv* kv, int32_t layer, int32_t start, int32_t len, const void* k_src,
                  const void* v_src, void* stream) {
  if (!kv || !k_src || !v_src) return fail(LOPA_EINVAL, "null pointer argument");
  const lopa_model_cfg& c = kv->m->cfg;
  if (layer < 0 || layer >= c.layers || start < 0 || len < 1 || (int64_t)start + len > kv->max_len)
    return fail(LOPA_EINVAL, "layer/start/len out of range");
  const int d = c.head_dim, Hkv = c.kv_heads;
  uint16_t* ck = kv->cache + ((size_t)layer * 2 + 0) * Hkv * d * kv->vld;
  uint16_t* cv = kv->cache + ((size_t)layer * 2 + 1) * Hkv * d * kv->vld;
  HIP_TRY(launch_kv_rows(ck, cv, (int64_t)d * kv->vld, kv->vld, Hkv, d, start, len,
                         (uint16_t*)k_src, (uint16_t*)v_src, 1, (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_kv_read_staging(const lopa_kv* kv, int32_t branch, int32_t layer, void* k_dst,
                         void* v_dst, void* stream) {
  if (!kv || !k_dst || !v_dst) return fail(LOPA_EINVAL, "null pointer argument");
  const lopa_model_cfg& c = kv->m->cfg;
  if (kv->last_nb < 0) return fail(LOPA_EINVAL, "nothing staged yet");
  if (branch < 0 || branch >= kv->last_nb || layer < 0 || layer >= c.layers)
    return fail(LOPA_EINVAL, "branch/layer out of range");
  const int d = c.head_dim, Hkv = c.kv_heads, L = kv->last_L;
  const size_t head = (size_t)d * kv->vlds;
  uint16_t* sk = kv->staging + (((size_t)branch * c.layers + layer) * 2 + 0) * Hkv * head;
  uint16_t* sv = kv->staging + (((size_t)branch * c.layers + layer) * 2 + 1) * Hkv * head;
  HIP_TRY(launch_kv_rows(sk, sv, (int64_t)head, kv->vlds, Hkv, d, 0, L, (uint16_t*)k_dst,
                         (uint16_t*)v_dst, 0, (hipStream_t)stream));
  return LOPA_OK;
}

int lopa_kv_set_block_causal(lopa_kv* kv, int32_t sub_block) {
  if (!kv) return fail(LOPA_EINVAL, "null pointer argument");
  if (sub_block < 0 || sub_block % 16)
    return fail(LOPA_EINVAL, "sub_block %d is not 0 or a positive multiple of 16", sub_block);
  kv->causal_blk = sub_block;
  return LOPA_OK;
}

int lopa_kv_profile(lopa_kv* kv, int32_t kinds_mask) {
  if (!kv) return fail(LOPA_EINVAL, "null pointer argument");
  if (kinds_mask < 0 || kinds_mask >= (1 << LOPA_PROF_KINDS)) return fail(LOPA_EINVAL, "bad mask");
  kv->prof_mask = kinds_mask;
  return LOPA_OK;
}

int lopa_kv_profile_read(lopa_kv* kv, double* total_ms, int64_t* launches) {
  if (!kv || !total_ms || !launches) return fail(LOPA_EINVAL, "null pointer argument");
  for (size_t i = 0; i < kv->ev_used; ++i) {
    lopa_kv::Ev& e = kv->ev_pool[i];
    HIP_TRY(hipEventSynchronize(e.b));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, e.a, e.b));
    kv->prof_ms[e.kind] += ms;
    kv->prof_n[e.kind] += 1;
  }
  kv->ev_used = 0;
  for (int k = 0; k < LOPA_PROF_KINDS; ++k) {
    total_ms[k] = kv->prof_ms[k];
    launches[k] = kv->prof_n[k];
    kv->prof_ms[k] = 0.0;
    kv->prof_n[k] = 0;
  }
  return LOPA_OK;
}

}  // extern "C"

// ------------------------------------------------- workspace (internal)
int model_device(const lopa_model* m) { return m->device; }

int lopa_fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int verify_check(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                 const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                 int32_t* pred) {
  if (!conf || !pred) return fail(LOPA_EINVAL, "null pointer argument");
  return check_verify(m, kv, prefix_len, branch_tokens, n_branches, L);
}

int verify_with_ws(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                   const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                   int32_t* pred, void* stream, const VerifyWs& ws) {
  return verify_impl(m, kv, prefix_len, branch_tokens, n_branches, L, conf, pred, stream, -1,
                     nullptr, ws);
}

namespace {
// the regions of a VerifyWs for nb x L rows, in carving order (bytes, each
// rounded up to 256): x, abuf, fbuf, qbuf, partials, pm, ps, pi, then the FP8
// operands of FP8 models
struct WsLayout {
  size_t sz[13] = {};
};
WsLayout ws_layout(const lopa_model* m, int32_t nb, int32_t L) {
  const lopa_model_cfg& c = m->cfg;
  const size_t rows = (size_t)padded_rows(nb * L);
  const int MT = (int)(rows / 256);
  const StepPlans p = step_plans(m, MT);
  WsLayout w;
  w.sz[0] = rows * c.hidden * 4;
  w.sz[1] = rows * c.hidden * 2;
  w.sz[2] = rows * round256(c.ffn) * 2;
  w.sz[3] = (size_t)nb * c.heads * L * c.head_dim * 2;
  w.sz[4] = std::max({(size_t)16, plan_partial_bytes(EPI_QKV, p.qkv, MT),
                      plan_partial_bytes(EPI_RESID, p.o, MT), plan_partial_bytes(EPI_RESID, p.down, MT),
                      attention_scratch_bytes(nb, L, c.heads, c.kv_heads, c.head_dim)});
  w.sz[5] = w.sz[6] = w.sz[7] = rows * m->tiles_lm * 4;
  if (m->fp8) {
    w.sz[8] = rows * round512(c.hidden);
    w.sz[9] = rows * round512(c.ffn);
    w.sz[10] = w.sz[11] = w.sz[12] = rows * 4;
  }
  for (size_t& v : w.sz) v = (v + 255) / 256 * 256;
  return w;
}
}  // namespace

size_t verify_ws_bytes(const lopa_model* m, int32_t n_branches, int32_t L) {
  size_t t = 0;
  for (size_t v : ws_layout(m, n_branches, L).sz) t += v;
  return t;
}

VerifyWs verify_ws_carve(const lopa_model* m, int32_t n_branches, int32_t L, char* base) {
  const WsLayout w = ws_layout(m, n_branches, L);
  char* r[13];
  for (int i = 0; i < 13; ++i) {
    r[i] = base;
    base += w.sz[i];
  }
  VerifyWs ws;
  ws.x = (float*)r[0];
  ws.abuf = (uint16_t*)r[1];
  ws.fbuf = (uint16_t*)r[2];
  ws.qbuf = (uint16_t*)r[3];
  ws.partials = (float*)r[4];
  ws.partials_bytes = w.sz[4];
  ws.pm = (float*)r[5];
  ws.ps = (float*)r[6];
  ws.pi = (int32_t*)r[7];
  if (m->fp8) {
    ws.a8_gu = (uint8_t*)r[8];
    ws.a8_dn = (uint8_t*)r[9];
    ws.sa_gu = (float*)r[10];
    ws.sa_dn = (float*)r[11];
    ws.rowmax_dn = (uint32_t*)r[12];
  }
  return ws;
}

int verify_ws_clear_padding(const lopa_model* m, int32_t n_branches, int32_t L, const VerifyWs& ws,
                            hipStream_t s) {
  // packed operands are [column block][row block] fragments, so a matrix's
  // padding columns are one contiguous tail: bf16 blocks of 32 columns x 16
  // rows (1 KiB), E4M3 blocks of 64 columns x 16 rows (1 KiB)
  const lopa_model_cfg& c = m->cfg;
  const size_t rb = (size_t)padded_rows(n_branches * L) / 16;
  auto tail = [&](void* buf, size_t cols, size_t padded, size_t per_block) -> hipError_t {
    if (padded == cols) return hipSuccess;
    const size_t from = cols / per_block * rb * 1024, to = padded / per_block * rb * 1024;
    return launch_fill_zero((char*)buf + from, to - from, s);
  };
  hipError_t e;
  if ((e = tail(ws.fbuf, c.ffn, round256(c.ffn), 32)) != hipSuccess ||
      (m->fp8 && ((e = tail(ws.a8_gu, c.hidden, round512(c.hidden), 64)) != hipSuccess ||
                  (e = tail(ws.a8_dn, c.ffn, round512(c.ffn), 64)) != hipSuccess)))
    return fail(LOPA_EHIP, "clearing the padding columns: %s", hipGetErrorString(e));
  return LOPA_OK;
}

// Branch construction (Eq. 1 + top-k, Alg. 1 steps 1-2), branch scoring and
// selection (Eq. 2, Alg. 1 step 3), and the winner's K/V commit (Sec. 3.4).
// Each runs as one small launch; the decision logic is integer work on fp32
// comparisons, done by one wavefront per block row.
#include "common.h"
#include "kernels.h"

#include <math.h>

// One workgroup of 256 threads; thread i owns window position i (L <= 256).
// Positions [0, n_elig) are eligible for the Eq. 1 fallback and the lookahead
// fills (all of them for one block; the fully activated blocks of a
// multi-block window).
__global__ __launch_bounds__(256) void build_branches_kernel(
    const int32_t* __restrict__ tokens, const float* __restrict__ conf,
    const int32_t* __restrict__ pred, int L, int n_elig, int mask_id, float tau, int k,
    int32_t* __restrict__ branch_tokens, int32_t* __restrict__ fill_pos,
    uint8_t* __restrict__ valid, int32_t* __restrict__ n_valid) {
  __shared__ float s_conf[256];
  __shared__ int s_rem[256];
  __shared__ float s_bc[4];
  __shared__ int s_bi[4];
  const int i = threadIdx.x, wv = i >> 6;
  const bool in = i < L;
  const int tok = in ? tokens[i] : 0;
  const float c = in ? conf[i] : 0.f;
  const int pr = in ? pred[i] : 0;
  const bool unf = in && tok == mask_id;

  // Eq. 1: S_high = {i in M_t : conf_i > tau}; else the argmax of conf over M_t.
  const bool high = unf && (c > tau);
  const bool any_high = __syncthreads_or(high) != 0;
  bool fill = high;
  if (!any_high) {
    // lowest position among the largest conf of the eligible unfilled set:
    // per wavefront, then over the four in order
    const bool el = unf && i < n_elig;
    float bc = el ? c : -INFINITY;
    int bi = el ? i : 0x7fffffff;
    for (int o = 32; o > 0; o >>= 1) {
      float oc = __shfl_xor(bc, o);
      int oi = __shfl_xor(bi, o);
      if (oc > bc || (oc == bc && oi < bi)) { bc = oc; bi = oi; }
    }
    if ((i & 63) == 0) {
      s_bc[wv] = bc;
      s_bi[wv] = bi;
    }
    __syncthreads();
    bc = s_bc[0];
    bi = s_bi[0];
    for (int w = 1; w < 4; ++w)
      if (s_bc[w] > bc || (s_bc[w] == bc && s_bi[w] < bi)) { bc = s_bc[w]; bi = s_bi[w]; }
    fill = (i == bi) && el;
  }
  const int b0 = fill ? pr : tok;
  const bool rem = in && i < n_elig && (b0 == mask_id);  // eligible part of M_B0

  // Rank of each position of M_B0 by (conf desc, position asc).
  s_conf[i] = c;
  s_rem[i] = rem ? 1 : 0;
  const int n_rem = __syncthreads_count(rem);
  int rank = 0;
  if (rem) {
    for (int j = 0; j < L; ++j) {
      if (!s_rem[j]) continue;
      const float cj = s_conf[j];
      rank += (cj > c || (cj == c && j < i)) ? 1 : 0;
    }
  }
  const int k_eff = k < n_rem ? k : n_rem;

  // Branch j: B0, plus position p_j (rank j-1) filled with pred.
  if (in) {
    for (int j = 0; j <= k; ++j) {
      int v = b0;
      if (rem && j >= 1 && rank == j - 1 && j <= k_eff) v = pr;
      branch_tokens[(int64_t)j * L + i] = v;
    }
  }
  if (rem && rank < k_eff) fill_pos[rank + 1] = i;
  for (int j = i; j <= k; j += 256) {
    if (j == 0 || j > k_eff) fill_pos[j] = -1;
    valid[j] = (j <= k_eff) ? 1 : 0;
  }
  if (i == 0) n_valid[0] = 1 + k_eff;
}

// Eq. 2 per branch (metric 0), or one of the alternative branch confidences
// named after it (Sec. 3.2): 1 = the smallest mean over runs of `window`
// consecutive unfilled positions (position order; all of them if fewer),
// 2 = the mean of the ceil(eta m) least confident unfilled positions (at
// least one). One wavefront per branch row, lane l holding positions l,
// l + 64, .. (L <= 256), with fixed reduction orders, so identical rows give
// bit-identical scores; then the argmax and the next state.
constexpr int SEL_CH = 4;  // position chunks of 64 per row
__global__ __launch_bounds__(256) void select_kernel(
    const int32_t* __restrict__ branch_tokens, const float* __restrict__ conf,
    const int32_t* __restrict__ pred, const uint8_t* __restrict__ valid, int nb, int L,
    int mask_id, int metric, int window, float eta, float* __restrict__ scores,
    int32_t* __restrict__ winner, int32_t* __restrict__ next_tokens,
    float* __restrict__ next_conf, int32_t* __restrict__ next_pred,
    int32_t* __restrict__ next_unfilled) {
  __shared__ float s_score[1024];
  __shared__ float s_row[4][64 * SEL_CH];
  __shared__ int s_win;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int nch = (L + 63) >> 6;  // chunks in use
  for (int j = wv; j < nb; j += 4) {
    bool m[SEL_CH];
    float c[SEL_CH];
    uint64_t bal[SEL_CH];
    int cnt = 0;
    float part = 0.f;  // this lane's unfilled conf, chunk order
#pragma unroll
    for (int q = 0; q < SEL_CH; ++q) {
      const int p = q * 64 + lane;
      const bool in = q < nch && p < L;
      const int t = in ? branch_tokens[(int64_t)j * L + p] : 0;
      m[q] = in && t == mask_id;
      c[q] = m[q] ? conf[(int64_t)j * L + p] : 0.f;
      bal[q] = __ballot(m[q]);
      cnt += __popcll(bal[q]);
      part += c[q];
    }
    float sc = INFINITY;
    if (cnt) {
      const float mean = wave_sum(part) / (float)cnt;
      sc = mean;
      if (metric == 1 && cnt > window) {
        // unfilled Conf compacted in position order, then each run start sums
        // its run in order
        int before = 0;
#pragma unroll
        for (int q = 0; q < SEL_CH; ++q) {
          const int rank = before + __popcll(bal[q] & ((1ull << lane) - 1ull));
          if (m[q]) s_row[wv][rank] = c[q];
          before += __popcll(bal[q]);
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        __builtin_amdgcn_wave_barrier();
        float v = INFINITY;
#pragma unroll
        for (int q = 0; q < SEL_CH; ++q) {
          const int r0 = q * 64 + lane;
          if (r0 <= cnt - window) {
            float acc = 0.f;
            for (int i = 0; i < window; ++i) acc += s_row[wv][r0 + i];
            v = fminf(v, acc / (float)window);
          }
        }
        sc = -wave_max(-v);
        __builtin_amdgcn_wave_barrier();
      } else if (metric == 2) {
        // rank in (Conf ascending, position ascending) order among the unfilled
#pragma unroll
        for (int q = 0; q < SEL_CH; ++q) s_row[wv][q * 64 + lane] = m[q] ? c[q] : INFINITY;
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
        const int kk = max(1, (int)ceil((double)eta * (double)cnt));
        float low = 0.f;
#pragma unroll
        for (int q = 0; q < SEL_CH; ++q) {
          const int p = q * 64 + lane;
          int rank = 0;
          for (int i = 0; i < L; ++i) {
            const float o = s_row[wv][i];
            rank += (o < c[q] || (o == c[q] && i < p)) ? 1 : 0;
          }
          low += (m[q] && rank < kk) ? c[q] : 0.f;
        }
        sc = wave_sum(low) / (float)kk;
        __builtin_amdgcn_wave_barrier();
      }
    }
    if (!valid[j]) sc = -INFINITY;
    if (lane == 0) {
      scores[j] = sc;
      s_score[j] = sc;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    for (int j = 1; j < nb; ++j)
      if (s_score[j] > s_score[best]) best = j;
    s_win = best;
    winner[0] = best;
  }
  __syncthreads();
  const int w = s_win;
  const int i = threadIdx.x;
  const bool in = i < L;
  int t = 0;
  if (in) {
    t = branch_tokens[(int64_t)w * L + i];
    next_tokens[i] = t;
    next_conf[i] = conf[(int64_t)w * L + i];
    next_pred[i] = pred[(int64_t)w * L + i];
  }
  const int cnt = __syncthreads_count(in && t == mask_id);
  if (i == 0) next_unfilled[0] = cnt;
}

// Copy n rows of the winner's staged K/V of one (layer, K/V, head) lhg into
// cache positions [P, P + n) (both in the KV tile layout of common.h; head
// regions d x vlds and d x vld elements). Whole tiles on both sides (P and n
// multiples of 32, the usual block commit) are one contiguous run; otherwise
// element by element.
__device__ __forceinline__ void commit_rows(const uint16_t* __restrict__ staging,
                                            uint16_t* __restrict__ cache, int w, int lhg,
                                            int layers, int Hkv, int vlds, int vld, int d, int P,
                                            int n) {
  const bool is_v = (lhg / Hkv) & 1;
  const uint16_t* src = staging + ((int64_t)w * layers * 2 * Hkv + lhg) * d * vlds;
  uint16_t* dst = cache + (int64_t)lhg * d * vld;
  if (((P | n) & (KV_TILE - 1)) == 0) {
    const uint4* s4 = (const uint4*)src;
    uint4* d4 = (uint4*)(dst + (int64_t)P * d);
    for (int e = threadIdx.x; e < n * d / 8; e += blockDim.x) d4[e] = s4[e];
    return;
  }
  for (int e = threadIdx.x; e < n * d; e += blockDim.x) {
    const int i = e / d, dim = e % d;
    if (is_v) dst[kv_v_off(P + i, dim, d)] = src[kv_v_off(i, dim, d)];
    else dst[kv_k_off(P + i, dim, d)] = src[kv_k_off(i, dim, d)];
  }
}

// The winner's staged K/V of every (layer, K/V, head) into cache positions
// [P, P + L). grid = layers * 2 * Hkv.
__global__ __launch_bounds__(256) void commit_kernel(
    const uint16_t* __restrict__ staging, uint16_t* __restrict__ cache,
    const int32_t* __restrict__ winner, int nb_last, int layers, int Hkv, int vlds, int vld,
    int d, int P, int L, int32_t* __restrict__ append_offset) {
  const int w = winner[0];
  const bool ok = (w >= 0 && w < nb_last);
  if (blockIdx.x == 0 && threadIdx.x == 0) append_offset[0] = ok ? P : -1;
  if (!ok) return;
  commit_rows(staging, cache, w, blockIdx.x, layers, Hkv, vlds, vld, d, P, L);
}

// ------------------------------------------------------- multi-block window
// The window state (lopa_window, device memory) after a selection: the gates
// of Sec. 3.3 in the library's readings, for the window tokens / conf / pred
// of the winner. One workgroup; the decisions are one thread's integer work
// on the blocks' filled counts, the moves of the window's rows are spread
// over the workgroup.
//   1. block b >= 1 becomes fully activated once block b - 1 is, and block
//      b - 1 has at least act_min filled positions (in block order);
//   2. the leading blocks with no masked position leave the window: their
//      tokens go to out (in order), their K/V are committed at the window's
//      prefix (lopa_window_commit, recorded in last_commit / last_commit_at),
//      the later rows move to the front, and the new first block is fully
//      activated;
//   3. an empty window with blocks still to generate opens one (fully
//      activated, need_initial = 1: its initial forward has not run); then
//      blocks are appended (not activated) while the window has room, blocks
//      remain, and the last block has at least add_min filled positions.
// Opened and appended blocks are all masked, conf 0, pred the mask token.
__global__ __launch_bounds__(256) void window_update_kernel(lopa_window* __restrict__ win,
                                                            int32_t* __restrict__ tokens,
                                                            float* __restrict__ conf,
                                                            int32_t* __restrict__ pred,
                                                            int32_t* __restrict__ out) {
  __shared__ int s_cnt[LOPA_WINDOW_MAX_BLOCKS];
  __shared__ int s_dec[4];  // moved blocks, blocks before / after, blocks committed before
  const int i = threadIdx.x;
  const int L = win->L, nw = win->blocks, mask = win->mask_id;
  const int Lw = nw * L;
  if (i < LOPA_WINDOW_MAX_BLOCKS) s_cnt[i] = 0;
  __syncthreads();
  const bool in = i < Lw;
  int tok = 0, pr = 0;
  float cf = 0.f;
  if (in) {
    tok = tokens[i];
    cf = conf[i];
    pr = pred[i];
    if (tok != mask) atomicAdd(&s_cnt[i / L], 1);
  }
  __syncthreads();
  if (i == 0) {
    int* cnt = s_cnt;  // this thread's from here on
    for (int b = 1; b < nw; ++b)
      if (!win->active[b] && win->active[b - 1] && cnt[b - 1] >= win->act_min) win->active[b] = 1;
    int c = 0;
    while (c < nw && cnt[c] == L) ++c;
    const int committed0 = win->committed;
    win->last_commit = c;
    win->last_commit_at = win->prefix_len;
    win->prefix_len += c * L;
    win->committed += c;
    int n2 = nw - c;
    for (int b = 0; b < n2; ++b) {
      win->active[b] = win->active[b + c];
      cnt[b] = cnt[b + c];
    }
    if (c && n2) win->active[0] = 1;
    int need = 0;
    if (n2 == 0 && win->added < win->n_blocks) {
      win->active[0] = 1;
      cnt[0] = 0;
      n2 = 1;
      ++win->added;
      need = 1;
    }
    while (n2 < win->w_max && win->added < win->n_blocks && cnt[n2 - 1] >= win->add_min) {
      win->active[n2] = 0;
      cnt[n2] = 0;
      ++n2;
      ++win->added;
    }
    for (int b = n2; b < LOPA_WINDOW_MAX_BLOCKS; ++b) win->active[b] = 0;
    int e = 0;
    while (e < n2 && win->active[e]) ++e;
    win->blocks = n2;
    win->eligible = e * L;
    win->need_initial = need;
    win->done = win->committed >= win->n_blocks ? 1 : 0;
    s_dec[0] = c;
    s_dec[1] = nw;
    s_dec[2] = n2;
    s_dec[3] = committed0;
  }
  __syncthreads();
  const int c = s_dec[0], n2 = s_dec[2], cl = c * L;
  if (in && i < cl) out[(int64_t)s_dec[3] * L + i] = tok;
  if (in && i >= cl) {
    tokens[i - cl] = tok;
    conf[i - cl] = cf;
    pred[i - cl] = pr;
  }
  for (int p = Lw - cl + i; p < n2 * L; p += blockDim.x) {
    tokens[p] = mask;
    conf[p] = 0.f;
    pred[p] = mask;
  }
}

// Header of a new window: no block yet; the first update opens block 0.
__global__ void window_init_kernel(lopa_window* __restrict__ win, int L, int w_max, int n_blocks,
                                   int prefix_len, int mask_id, int add_min, int act_min) {
  if (threadIdx.x == 0) {
    win->blocks = 0;
    win->eligible = 0;
    win->prefix_len = prefix_len;
    win->need_initial = 0;
    win->done = n_blocks <= 0 ? 1 : 0;
    win->added = 0;
    win->committed = 0;
    win->last_commit = 0;
    win->last_commit_at = prefix_len;
    win->error = 0;
    win->L = L;
    win->w_max = w_max;
    win->n_blocks = n_blocks;
    win->mask_id = mask_id;
    win->add_min = add_min;
    win->act_min = act_min;
  }
  if (threadIdx.x < LOPA_WINDOW_MAX_BLOCKS) win->active[threadIdx.x] = 0;
}

// The K/V of the blocks the last window update committed (last_commit blocks
// of L rows, at last_commit_at): the winner's staged rows [0, n) of the
// last verify forward (n <= last_L rows, committing up to max_len).
__global__ __launch_bounds__(256) void window_commit_kernel(
    const uint16_t* __restrict__ staging, uint16_t* __restrict__ cache,
    const int32_t* __restrict__ winner, lopa_window* __restrict__ win, int nb_last, int last_L,
    int max_len, int layers, int Hkv, int vlds, int vld, int d) {
  const int w = winner[0];
  const int n = win->last_commit * win->L, P = win->last_commit_at;
  const bool ok = w >= 0 && w < nb_last && n >= 0 && n <= last_L && P >= 0 && P + n <= max_len;
  if (!ok) {
    if (blockIdx.x == 0 && threadIdx.x == 0) win->error = 1;
    return;
  }
  if (n == 0) return;
  commit_rows(staging, cache, w, blockIdx.x, layers, Hkv, vlds, vld, d, P, n);
}

// Positions [start, start + len) of one layer's K and V between the cache
// side (heads head_stride apart, KV tile layout) and a caller buffer
// [Hkv][len][d]. One workgroup per (head, K/V).
__global__ __launch_bounds__(256) void kv_rows_kernel(uint16_t* __restrict__ ck,
                                                      uint16_t* __restrict__ cv,
                                                      int64_t head_stride, int d,
                                                      int start, int len,
                                                      uint16_t* __restrict__ bk,
                                                      uint16_t* __restrict__ bv, int to_cache) {
  const int head = blockIdx.x >> 1, is_v = blockIdx.x & 1;
  uint16_t* c = (is_v ? cv : ck) + (int64_t)head * head_stride;
  uint16_t* b = (is_v ? bv : bk) + (int64_t)head * len * d;
  for (int e = threadIdx.x; e < len * d; e += blockDim.x) {
    const int i = e / d, dim = e % d;  // buffer element (i, dim)
    const int64_t co = is_v ? kv_v_off(start + i, dim, d) : kv_k_off(start + i, dim, d);
    if (to_cache) c[co] = b[e];
    else b[e] = c[co];
  }
}

// ------------------------------------------------------------ launchers
hipError_t launch_build_branches(const int32_t* tokens, const float* conf, const int32_t* pred,
                                 int L, int n_elig, int mask_id, float tau, int k,
                                 int32_t* branch_tokens, int32_t* fill_pos, uint8_t* valid,
                                 int32_t* n_valid, hipStream_t s) {
  if (L < 1 || L > 256 || n_elig < 1 || n_elig > L) return hipErrorInvalidValue;
  hipLaunchKernelGGL(build_branches_kernel, dim3(1), dim3(256), 0, s, tokens, conf, pred, L,
                     n_elig, mask_id, tau, k, branch_tokens, fill_pos, valid, n_valid);
  return hipGetLastError();
}

hipError_t launch_select(const int32_t* bt, const float* conf, const int32_t* pred,
                         const uint8_t* valid, int nb, int L, int mask_id, int metric,
                         int window, float eta, float* scores, int32_t* winner, int32_t* nt,
                         float* nc, int32_t* np, int32_t* nu, hipStream_t s) {
  if (nb < 1 || nb > 1024 || L < 1 || L > 64 * SEL_CH || metric < 0 || metric > 2 ||
      (metric == 1 && window < 1) || (metric == 2 && !(eta > 0.f && eta <= 1.f)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(256), 0, s, bt, conf, pred, valid, nb, L,
                     mask_id, metric, window, eta, scores, winner, nt, nc, np, nu);
  return hipGetLastError();
}

hipError_t launch_commit(const uint16_t* staging, uint16_t* cache, const int32_t* winner,
                         int nb_last, int layers, int Hkv, int vlds, int vld, int d, int P,
                         int L, int32_t* append_offset, hipStream_t s) {
  hipLaunchKernelGGL(commit_kernel, dim3(layers * 2 * Hkv), dim3(256), 0, s, staging, cache,
                     winner, nb_last, layers, Hkv, vlds, vld, d, P, L, append_offset);
  return hipGetLastError();
}

hipError_t launch_window_init(lopa_window* win, int L, int w_max, int n_blocks, int prefix_len,
                              int mask_id, int add_min, int act_min, hipStream_t s) {
  hipLaunchKernelGGL(window_init_kernel, dim3(1), dim3(64), 0, s, win, L, w_max, n_blocks,
                     prefix_len, mask_id, add_min, act_min);
  return hipGetLastError();
}

hipError_t launch_window_update(lopa_window* win, int32_t* tokens, float* conf, int32_t* pred,
                                int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(window_update_kernel, dim3(1), dim3(256), 0, s, win, tokens, conf, pred, out);
  return hipGetLastError();
}

hipError_t launch_window_commit(const uint16_t* staging, uint16_t* cache, const int32_t* winner,
                                lopa_window* win, int nb_last, int last_L, int max_len,
                                int layers, int Hkv, int vlds, int vld, int d, hipStream_t s) {
  hipLaunchKernelGGL(window_commit_kernel, dim3(layers * 2 * Hkv), dim3(256), 0, s, staging,
                     cache, winner, win, nb_last, last_L, max_len, layers, Hkv, vlds, vld, d);
  return hipGetLastError();
}

hipError_t launch_kv_rows(uint16_t* cache_k, uint16_t* cache_v, int64_t head_stride, int ld,
                          int Hkv, int d, int start, int len, uint16_t* buf_k, uint16_t* buf_v,
                          int to_cache, hipStream_t s) {
  if (ld % KV_TILE || start < 0 || start + len > ld) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kv_rows_kernel, dim3(2 * Hkv), dim3(256), 0, s, cache_k, cache_v,
                     head_stride, d, start, len, buf_k, buf_v, to_cache);
  return hipGetLastError();
}

// Branch construction (Eq. 1 + top-k, Alg. 1 steps 1-2), branch scoring and
// selection (Eq. 2, Alg. 1 step 3), and the winner's K/V commit (Sec. 3.4).
// Each runs as one small launch; the decision logic is integer work on fp32
// comparisons, done by one wavefront per block row.
#include "common.h"
#include "kernels.h"

#include <math.h>

// One wavefront (64 lanes), lane i owns block position i (L <= 64). Positions
// [0, n_elig) are eligible for the Eq. 1 fallback and the lookahead fills (all
// of them for one block; the fully activated blocks of a multi-block window).
__global__ __launch_bounds__(64) void build_branches_kernel(
    const int32_t* __restrict__ tokens, const float* __restrict__ conf,
    const int32_t* __restrict__ pred, int L, int n_elig, int mask_id, float tau, int k,
    int32_t* __restrict__ branch_tokens, int32_t* __restrict__ fill_pos,
    uint8_t* __restrict__ valid, int32_t* __restrict__ n_valid) {
  __shared__ float s_conf[64];
  __shared__ int s_rem[64];
  const int i = threadIdx.x;
  const bool in = i < L;
  const int tok = in ? tokens[i] : 0;
  const float c = in ? conf[i] : 0.f;
  const int pr = in ? pred[i] : 0;
  const bool unf = in && tok == mask_id;

  // Eq. 1: S_high = {i in M_t : conf_i > tau}; else the argmax of conf over M_t.
  const bool high = unf && (c > tau);
  const bool any_high = __ballot(high) != 0ull;
  bool fill = high;
  if (!any_high) {
    // lowest position among the largest conf of the eligible unfilled set
    const bool el = unf && i < n_elig;
    float bc = el ? c : -INFINITY;
    int bi = el ? i : 0x7fffffff;
    for (int o = 32; o > 0; o >>= 1) {
      float oc = __shfl_xor(bc, o);
      int oi = __shfl_xor(bi, o);
      if (oc > bc || (oc == bc && oi < bi)) { bc = oc; bi = oi; }
    }
    fill = (i == bi) && el;
  }
  const int b0 = fill ? pr : tok;
  const bool rem = in && i < n_elig && (b0 == mask_id);  // eligible part of M_B0

  // Rank of each position of M_B0 by (conf desc, position asc).
  s_conf[i] = c;
  s_rem[i] = rem ? 1 : 0;
  __syncthreads();
  int rank = 0;
  if (rem) {
    for (int j = 0; j < L; ++j) {
      if (!s_rem[j]) continue;
      const float cj = s_conf[j];
      rank += (cj > c || (cj == c && j < i)) ? 1 : 0;
    }
  }
  const int n_rem = __popcll(__ballot(rem));
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
  for (int j = i; j <= k; j += 64) {
    if (j == 0 || j > k_eff) fill_pos[j] = -1;
    valid[j] = (j <= k_eff) ? 1 : 0;
  }
  if (i == 0) n_valid[0] = 1 + k_eff;
}

// Eq. 2 per branch (metric 0), or one of the alternative branch confidences
// named after it (Sec. 3.2): 1 = the smallest mean over runs of `window`
// consecutive unfilled positions (position order; all of them if fewer),
// 2 = the mean of the ceil(eta m) least confident unfilled positions (at
// least one). One wavefront per branch row with fixed reduction orders, so
// identical rows give bit-identical scores; then the argmax and the next state.
__global__ __launch_bounds__(256) void select_kernel(
    const int32_t* __restrict__ branch_tokens, const float* __restrict__ conf,
    const int32_t* __restrict__ pred, const uint8_t* __restrict__ valid, int nb, int L,
    int mask_id, int metric, int window, float eta, float* __restrict__ scores,
    int32_t* __restrict__ winner, int32_t* __restrict__ next_tokens,
    float* __restrict__ next_conf, int32_t* __restrict__ next_pred,
    int32_t* __restrict__ next_unfilled) {
  __shared__ float s_score[1024];
  __shared__ float s_row[4][64];
  __shared__ int s_win;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int j = wv; j < nb; j += 4) {
    const bool in = lane < L;
    const int t = in ? branch_tokens[(int64_t)j * L + lane] : 0;
    const bool m = in && t == mask_id;
    const float c = m ? conf[(int64_t)j * L + lane] : 0.f;
    const uint64_t bal = __ballot(m);
    const int cnt = __popcll(bal);
    float sc = INFINITY;
    if (cnt) {
      const float mean = wave_sum(c) / (float)cnt;
      sc = mean;
      if (metric == 1 && cnt > window) {
        // unfilled Conf compacted in position order, then each run start sums
        // its run in order
        const int rank = __popcll(bal & ((1ull << lane) - 1ull));
        if (m) s_row[wv][rank] = c;
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        __builtin_amdgcn_wave_barrier();
        float v = INFINITY;
        if (lane <= cnt - window) {
          float acc = 0.f;
          for (int i = 0; i < window; ++i) acc += s_row[wv][lane + i];
          v = acc / (float)window;
        }
        sc = -wave_max(-v);
        __builtin_amdgcn_wave_barrier();
      } else if (metric == 2) {
        // rank in (Conf ascending, position ascending) order among the unfilled
        s_row[wv][lane] = m ? c : INFINITY;
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
        int rank = 0;
        for (int i = 0; i < L; ++i) {
          const float o = s_row[wv][i];
          rank += (o < c || (o == c && i < lane)) ? 1 : 0;
        }
        const int kk = max(1, (int)ceil((double)eta * (double)cnt));
        sc = wave_sum(m && rank < kk ? c : 0.f) / (float)kk;
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
  if (threadIdx.x < 64) {
    const int i = threadIdx.x;
    const bool in = i < L;
    int t = 0;
    if (in) {
      t = branch_tokens[(int64_t)w * L + i];
      next_tokens[i] = t;
      next_conf[i] = conf[(int64_t)w * L + i];
      next_pred[i] = pred[(int64_t)w * L + i];
    }
    const int cnt = __popcll(__ballot(in && t == mask_id));
    if (i == 0) next_unfilled[0] = cnt;
  }
}

// Copy the winner's staged K/V of every (layer, K/V, head) into cache
// positions [P, P + L). grid = layers * 2 * Hkv; the layouts are the KV
// layouts of kernels.h (V transposed, leading dimensions vlds / vld).
__global__ __launch_bounds__(256) void commit_kernel(
    const uint16_t* __restrict__ staging, uint16_t* __restrict__ cache,
    const int32_t* __restrict__ winner, int nb_last, int layers, int Hkv, int vlds, int vld,
    int d, int P, int L, int32_t* __restrict__ append_offset) {
  const int w = winner[0];
  const bool ok = (w >= 0 && w < nb_last);
  if (blockIdx.x == 0 && threadIdx.x == 0) append_offset[0] = ok ? P : -1;
  if (!ok) return;
  const int lhg = blockIdx.x;  // (layer, kv, head) flattened
  const bool is_v = (lhg / Hkv) & 1;
  const uint16_t* src = staging + ((int64_t)w * layers * 2 * Hkv + lhg) * d * vlds;
  uint16_t* dst = cache + (int64_t)lhg * d * vld;
  if (!is_v) {
    const uint4* s4 = (const uint4*)src;
    uint4* d4 = (uint4*)(dst + (int64_t)P * d);
    for (int e = threadIdx.x; e < L * d / 8; e += blockDim.x) d4[e] = s4[e];
  } else if (L <= 256) {
    // V^T rows: dimension dim holds its L positions contiguously. With lp the
    // power of two >= L, thread t copies position t % lp of dimensions
    // t / lp, t / lp + 256 / lp, ... (shifts and masks, no division)
    const int lg = 32 - __builtin_clz(L - 1 > 0 ? L - 1 : 1) - (L == 1 ? 1 : 0);
    const int i = threadIdx.x & ((1 << lg) - 1);
    if (i < L)
      for (int dim = threadIdx.x >> lg; dim < d; dim += 256 >> lg)
        dst[(int64_t)dim * vld + P + i] = src[(int64_t)dim * vlds + i];
  } else {
    for (int e = threadIdx.x; e < L * d; e += blockDim.x) {
      const int dim = e / L, i = e % L;
      dst[(int64_t)dim * vld + P + i] = src[(int64_t)dim * vlds + i];
    }
  }
}

// Positions [start, start + len) of one layer's K and V between the cache
// side (heads head_stride apart; K [pos][d], V [d][ld]) and a caller buffer
// [Hkv][len][d]. One workgroup per (head, K/V).
__global__ __launch_bounds__(256) void kv_rows_kernel(uint16_t* __restrict__ ck,
                                                      uint16_t* __restrict__ cv,
                                                      int64_t head_stride, int ld, int d,
                                                      int start, int len,
                                                      uint16_t* __restrict__ bk,
                                                      uint16_t* __restrict__ bv, int to_cache) {
  const int head = blockIdx.x >> 1, is_v = blockIdx.x & 1;
  uint16_t* c = (is_v ? cv : ck) + (int64_t)head * head_stride;
  uint16_t* b = (is_v ? bv : bk) + (int64_t)head * len * d;
  for (int e = threadIdx.x; e < len * d; e += blockDim.x) {
    const int i = e / d, dim = e % d;  // buffer element (i, dim)
    const int64_t co = is_v ? (int64_t)dim * ld + start + i : (int64_t)(start + i) * d + dim;
    if (to_cache) c[co] = b[e];
    else b[e] = c[co];
  }
}

// ------------------------------------------------------------ launchers
hipError_t launch_build_branches(const int32_t* tokens, const float* conf, const int32_t* pred,
                                 int L, int n_elig, int mask_id, float tau, int k,
                                 int32_t* branch_tokens, int32_t* fill_pos, uint8_t* valid,
                                 int32_t* n_valid, hipStream_t s) {
  if (L < 1 || L > 64 || n_elig < 1 || n_elig > L) return hipErrorInvalidValue;
  hipLaunchKernelGGL(build_branches_kernel, dim3(1), dim3(64), 0, s, tokens, conf, pred, L,
                     n_elig, mask_id, tau, k, branch_tokens, fill_pos, valid, n_valid);
  return hipGetLastError();
}

hipError_t launch_select(const int32_t* bt, const float* conf, const int32_t* pred,
                         const uint8_t* valid, int nb, int L, int mask_id, int metric,
                         int window, float eta, float* scores, int32_t* winner, int32_t* nt,
                         float* nc, int32_t* np, int32_t* nu, hipStream_t s) {
  if (nb < 1 || nb > 1024 || L < 1 || L > 64 || metric < 0 || metric > 2 ||
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

hipError_t launch_kv_rows(uint16_t* cache_k, uint16_t* cache_v, int64_t head_stride, int ld,
                          int Hkv, int d, int start, int len, uint16_t* buf_k, uint16_t* buf_v,
                          int to_cache, hipStream_t s) {
  hipLaunchKernelGGL(kv_rows_kernel, dim3(2 * Hkv), dim3(256), 0, s, cache_k, cache_v,
                     head_stride, ld, d, start, len, buf_k, buf_v, to_cache);
  return hipGetLastError();
}

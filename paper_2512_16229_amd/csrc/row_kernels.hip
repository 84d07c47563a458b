// Row-wise kernels of the verify forward: embedding gather + RMSNorm, RMSNorm
// into the packed GEMM operand, the merge of the LM head's per-tile softmax
// partials into Conf / candidate token (Sec. 3.1), and the one-time weight
// repacking.
#include "common.h"
#include "kernels.h"

#include <math.h>

// Block-wide sum in a fixed order (wave butterfly, then waves in index order).
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) red[wv] = v;
  __syncthreads();
  float t = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return t;
}

// One workgroup per row. H % 128 == 0, so H/8 groups of 8 columns.
template <bool EMBED>
__global__ __launch_bounds__(256) void norm_kernel(const int32_t* __restrict__ tokens,
                                                   const uint16_t* __restrict__ embed, int vocab,
                                                   const float* __restrict__ w, float eps, int Mp,
                                                   int H, float* __restrict__ x,
                                                   uint16_t* __restrict__ a) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  float* xr = x + (int64_t)r * H;
  const int groups = H >> 3;
  float ss = 0.f;
  if (EMBED) {
    // a token outside [0, vocab) reads row 0 instead of memory past the table
    int tok = tokens[r];
    tok = (tok >= 0 && tok < vocab) ? tok : 0;
    const uint16_t* er = embed + (int64_t)tok * H;
    for (int gi = threadIdx.x; gi < groups; gi += 256) {
      uint4 raw = *(const uint4*)(er + gi * 8);
      const uint16_t* h = (const uint16_t*)&raw;
      float v[8];
      for (int e = 0; e < 8; ++e) {
        v[e] = bf2f_bits(h[e]);
        ss += v[e] * v[e];
      }
      *(float4*)(xr + gi * 8) = make_float4(v[0], v[1], v[2], v[3]);
      *(float4*)(xr + gi * 8 + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
  } else {
    for (int gi = threadIdx.x; gi < groups; gi += 256) {
      float4 p = *(const float4*)(xr + gi * 8), q = *(const float4*)(xr + gi * 8 + 4);
      ss += p.x * p.x + p.y * p.y + p.z * p.z + p.w * p.w + q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
    }
  }
  const float tot = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int gi = threadIdx.x; gi < groups; gi += 256) {
    float4 p = *(const float4*)(xr + gi * 8), q = *(const float4*)(xr + gi * 8 + 4);
    float v[8] = {p.x, p.y, p.z, p.w, q.x, q.y, q.z, q.w};
    uint16_t o[8];
    for (int e = 0; e < 8; ++e) o[e] = f2bf_bits(v[e] * inv * w[gi * 8 + e]);
    *(uint4*)(a + packA_off(r, gi * 8, Mp)) = *(const uint4*)o;
  }
}

// One wavefront per row: merge (max, sum, argmax) of all vocabulary tiles.
__global__ __launch_bounds__(256) void lm_merge_kernel(const float* __restrict__ pm,
                                                       const float* __restrict__ ps,
                                                       const int32_t* __restrict__ pi, int M,
                                                       int tiles, float* __restrict__ conf,
                                                       int32_t* __restrict__ pred) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= M) return;
  float m = -INFINITY, s = 0.f;
  int idx = 0x7fffffff;
  for (int t = lane; t < tiles; t += 64) {
    const float tm = pm[(int64_t)r * tiles + t], ts = ps[(int64_t)r * tiles + t];
    const int ti = pi[(int64_t)r * tiles + t];
    if (tm == -INFINITY) continue;
    if (tm > m) {
      s = s * expf(m - tm) + ts;
      m = tm;
      idx = ti;
    } else {
      s += ts * expf(tm - m);
      if (tm == m && ti < idx) idx = ti;
    }
  }
  for (int o = 1; o < 64; o <<= 1) {
    const float om = __shfl_xor(m, o), os = __shfl_xor(s, o);
    const int oi = __shfl_xor(idx, o);
    const float nm = fmaxf(m, om);
    const float a = (m == -INFINITY) ? 0.f : s * expf(m - nm);
    const float b = (om == -INFINITY) ? 0.f : os * expf(om - nm);
    int ni;
    if (m > om) ni = idx;
    else if (om > m) ni = oi;
    else ni = idx < oi ? idx : oi;
    m = nm;
    s = a + b;
    idx = ni;
  }
  if (lane == 0) {
    conf[r] = 1.0f / s;
    pred[r] = (idx == 0x7fffffff) ? 0 : idx;  // all logits non-finite: report token 0
  }
}

// Weight repack: one thread per (fragment, lane) writes 8 bf16 (16 bytes);
// thread order is the packed order [block][kc][kk][lane].
__global__ __launch_bounds__(256) void repack_kernel(const uint16_t* __restrict__ s0, int r0,
                                                     const uint16_t* __restrict__ s1, int r1,
                                                     const uint16_t* __restrict__ s2, int r2,
                                                     int K, int KC, int64_t total, int pairs,
                                                     uint16_t* __restrict__ dst) {
  // K: length of a source row; KC * 64 >= K: packed columns, the excess is zero
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= total) return;
  const int lane = (int)(gid & 63);
  const int64_t u = gid >> 6;
  const int kk = (int)(u & 1);
  const int kc = (int)((u >> 1) % KC);
  const int blk = (int)((u >> 1) / KC);
  const int k0 = kc * 64 + kk * 32 + (lane >> 4) * 8;
  const uint16_t* src = nullptr;
  int row = 0;
  if (pairs) {
    row = (blk >> 1) * 16 + (lane & 15);
    if (!(blk & 1)) { if (row < r0) src = s0; }
    else { if (row < r1) src = s1; }
  } else {
    const int n = blk * 16 + (lane & 15);
    if (n < r0) { src = s0; row = n; }
    else if (n < r0 + r1) { src = s1; row = n - r0; }
    else if (n < r0 + r1 + r2) { src = s2; row = n - r0 - r1; }
  }
  uint4 v = make_uint4(0, 0, 0, 0);
  if (src && k0 < K) v = *(const uint4*)(src + (int64_t)row * K + k0);
  *(uint4*)(dst + gid * 8) = v;
}

__global__ void bf16_to_f32_kernel(const uint16_t* __restrict__ s, float* __restrict__ d, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) d[i] = bf2f_bits(s[i]);
}

// ------------------------------------------------------------ launchers
hipError_t launch_embed_norm(const int32_t* tokens, const uint16_t* embed, int vocab,
                             const float* w, float eps, int M, int Mp, int H, float* x,
                             uint16_t* a, hipStream_t s) {
  hipLaunchKernelGGL(norm_kernel<true>, dim3(M), dim3(256), 0, s, tokens, embed, vocab, w, eps, Mp,
                     H, x, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_pack(const float* x, const float* w, float eps, int M, int Mp, int H,
                               uint16_t* a, hipStream_t s) {
  hipLaunchKernelGGL(norm_kernel<false>, dim3(M), dim3(256), 0, s, nullptr, nullptr, 0, w, eps,
                     Mp, H, const_cast<float*>(x), a);
  return hipGetLastError();
}

hipError_t launch_lm_merge(const float* pm, const float* ps, const int32_t* pi, int M, int tiles,
                           float* conf, int32_t* pred, hipStream_t s) {
  hipLaunchKernelGGL(lm_merge_kernel, dim3((M + 3) / 4), dim3(256), 0, s, pm, ps, pi, M, tiles,
                     conf, pred);
  return hipGetLastError();
}

hipError_t launch_repack(const uint16_t* s0, int r0, const uint16_t* s1, int r1,
                         const uint16_t* s2, int r2, int K, int KP, int blocks, int pairs,
                         uint16_t* dst, hipStream_t s) {
  if (KP % 256 || KP < K) return hipErrorInvalidValue;
  const int KC = KP / 64;
  const int64_t total = (int64_t)blocks * KC * 2 * 64;
  const int64_t grid = (total + 255) / 256;
  hipLaunchKernelGGL(repack_kernel, dim3((unsigned)grid), dim3(256), 0, s, s0, r0, s1, r1, s2,
                     r2, K, KC, total, pairs, dst);
  return hipGetLastError();
}


hipError_t launch_bf16_to_f32(const uint16_t* src, float* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

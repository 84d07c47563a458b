// Row-wise kernels of the verify forward: embedding gather + RMSNorm, RMSNorm
// into the packed GEMM operand, the merge of the LM head's per-tile softmax
// partials into Conf / candidate token (Sec. 3.1), and the one-time weight
// repacking.
#include "common.h"
#include "kernels.h"

#include <math.h>

// One workgroup of TPB threads (256, 512 or 1024: the launcher takes the
// fewest that cover the row once, so a row's loads are spread over up to 16
// wavefronts) per row; thread t holds the 4-column groups q = t + TPB i,
// i < NG (columns 4 q .. 4 q + 3, q < H / 4, H % 256 == 0, H <= TPB NG 4).
// The row is formed in registers:
//   EMBED:  x = embedding of the token (bf16 -> fp32)
//   else:   x += sum of the S split-K partial sums of the preceding projection
//           (row-major fp32 [S][Mp][H], summed in split order first)
// then x is stored back and a = pack(x / rms(x) * w) (RMSNorm; the sum of
// squares is reduced in a fixed order: lanes, then wavefronts 0, 1, ...). Groups
// past the row read the row's last group again and are discarded by a
// select: no load sits under a branch, so all of them can be in flight
// together.
constexpr int H_MAX = 8192;  // widest row: 1024 threads x 2 groups of 4 columns

// E4M3 (no infinities, max 448) of x, round to nearest even, saturating:
// subnormals (|x| < 2^-6) are multiples of 2^-9, and a normal value of binade
// 2^E has 3 fraction bits, so its code is rint(|x| 2^(3 - E)) - 8 + (E + 7) 8
// (a mantissa that rounds up to 16 carries into the exponent by itself).
__device__ __forceinline__ uint32_t f32_to_e4m3(float x) {
  const uint32_t sign = (__float_as_uint(x) >> 24) & 0x80u;
  const float ax = fminf(fabsf(x), 448.f);
  if (ax < 0.015625f) return sign | (uint32_t)rintf(ax * 512.f);
  const int E = (int)((__float_as_uint(ax) >> 23) & 0xffu) - 127;
  return sign | (uint32_t)(((E + 7) << 3) + (int)rintf(ldexpf(ax, 3 - E)) - 8);
}
// byte offset of (row r, column c) in the packed FP8 operand: 64-column blocks
// of 16-row blocks, lane (r % 16) + 16 ((c % 64) / 16) holding 16 consecutive
// columns (the bf16 layout with twice the columns per lane slot)
__device__ __forceinline__ int64_t packA8_off(int r, int c, int Mp) {
  return ((int64_t)((c >> 6) * (Mp >> 4) + (r >> 4)) * 64 + (r & 15) + 16 * ((c & 63) >> 4)) * 16 +
         (c & 15);
}
// the per-row scaling of the FP8 operand: inverse 448 / max|v|, scale max|v| / 448
__device__ __forceinline__ float e4m3_inv(float amax) { return amax > 0.f ? __fdiv_rn(448.f, amax) : 0.f; }
__device__ __forceinline__ float e4m3_scale(float amax) { return amax > 0.f ? __fdiv_rn(amax, 448.f) : 0.f; }

template <bool EMBED, int SC, int NG, bool A8, int TPB>
__global__ __launch_bounds__(TPB) void resnorm_kernel(const int32_t* __restrict__ tokens,
                                                      const uint16_t* __restrict__ embed,
                                                      int vocab, const float* __restrict__ part,
                                                      int S, const float* __restrict__ w,
                                                      float eps, int M, int Mp, int H,
                                                      float* __restrict__ x,
                                                      uint16_t* __restrict__ a,
                                                      uint8_t* __restrict__ a8,
                                                      float* __restrict__ sa,
                                                      uint32_t* __restrict__ rowmax_zero) {
  constexpr int NW = TPB / 64;
  __shared__ float red[NW];
  __shared__ float redm[NW];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int r = blockIdx.x;
  const int nq = H >> 2;
  float* xr = x + (int64_t)r * H;
  float4 v[NG];
  float ss = 0.f;
  // the norm weights are loaded first, with the row's inputs, so that no
  // load waits behind the reduction
  float4 wt[NG];
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    const int q = tid + TPB * i;
    wt[i] = ((const float4*)w)[q < nq ? q : nq - 1];
  }
  if (EMBED) {
    // a token outside [0, vocab) reads row 0 instead of memory past the table
    int tok = tokens[r];
    tok = (tok >= 0 && tok < vocab) ? tok : 0;
    const uint16_t* er = embed + (int64_t)tok * H;
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      const bool ok = q < nq;
      const uint2 raw = *(const uint2*)(er + (ok ? q : nq - 1) * 4);
      v[i] = make_float4(ok ? bf2f_bits(raw.x & 0xffff) : 0.f, ok ? bf2f_bits(raw.x >> 16) : 0.f,
                         ok ? bf2f_bits(raw.y & 0xffff) : 0.f, ok ? bf2f_bits(raw.y >> 16) : 0.f);
    }
  } else {
    // partial sums in split order, then the residual. SC >= 0: the split count
    // is a compile-time constant; SC < 0: S, known at run time.
    float4 t[NG], res[NG];
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      res[i] = ((const float4*)xr)[q < nq ? q : nq - 1];  // the residual, loaded up front
      t[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    auto add_split = [&](int sp) {
      const float4* pr = (const float4*)(part + ((int64_t)sp * Mp + r) * H);
#pragma unroll
      for (int i = 0; i < NG; ++i) {
        const int q = tid + TPB * i;
        const float4 u = pr[q < nq ? q : nq - 1];
        t[i].x += u.x; t[i].y += u.y; t[i].z += u.z; t[i].w += u.w;
      }
    };
    if constexpr (SC >= 0) {
      // unrolled: every split's loads are issued before the first add
#pragma unroll
      for (int sp = 0; sp < SC; ++sp) add_split(sp);
    } else {
      for (int sp = 0; sp < S; ++sp) add_split(sp);
    }
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      const bool ok = q < nq;
      const float4 u = res[i];
      v[i] = make_float4(ok ? u.x + t[i].x : 0.f, ok ? u.y + t[i].y : 0.f,
                         ok ? u.z + t[i].z : 0.f, ok ? u.w + t[i].w : 0.f);
    }
  }
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    const int q = tid + TPB * i;
    if (q < nq && (EMBED || (SC >= 0 ? SC : S) > 0)) ((float4*)xr)[q] = v[i];
    ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
  }
  ss = wave_sum(ss);
  if (lane == 0) red[wv] = ss;
  __syncthreads();
  float tot = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  if constexpr (A8) {
    // FP8 operand: the normed row, its largest magnitude (lanes, then
    // wavefronts 0, 1, ...), then E4M3 of each value times 448 / max
    float4 y[NG];
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      y[i] = make_float4(v[i].x * inv * wt[i].x, v[i].y * inv * wt[i].y, v[i].z * inv * wt[i].z,
                         v[i].w * inv * wt[i].w);
      if (q < nq)
        mx = fmaxf(mx, fmaxf(fmaxf(fabsf(y[i].x), fabsf(y[i].y)), fmaxf(fabsf(y[i].z), fabsf(y[i].w))));
    }
    mx = wave_max(mx);
    if (lane == 0) redm[wv] = mx;
    __syncthreads();
    mx = redm[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) mx = fmaxf(mx, redm[w]);
    const float si = e4m3_inv(mx);
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      if (q < nq) {
        const uint32_t b = f32_to_e4m3(y[i].x * si) | (f32_to_e4m3(y[i].y * si) << 8) |
                           (f32_to_e4m3(y[i].z * si) << 16) | (f32_to_e4m3(y[i].w * si) << 24);
        *(uint32_t*)(a8 + packA8_off(r, q * 4, Mp)) = b;
      }
    }
    if (tid == 0) {
      sa[r] = e4m3_scale(mx);
      if (rowmax_zero) rowmax_zero[r] = 0u;  // for the SwiGLU GEMM's row maxima
    }
  } else {
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int q = tid + TPB * i;
      if (q < nq) {
        const uint32_t lo = (uint32_t)f2bf_bits(v[i].x * inv * wt[i].x) |
                            ((uint32_t)f2bf_bits(v[i].y * inv * wt[i].y) << 16);
        const uint32_t hi = (uint32_t)f2bf_bits(v[i].z * inv * wt[i].z) |
                            ((uint32_t)f2bf_bits(v[i].w * inv * wt[i].w) << 16);
        *(uint2*)(a + packA_off(r, q * 4, Mp)) = make_uint2(lo, hi);
      }
    }
  }
}

// FP8 operand of a projection from the packed bf16 one (the SwiGLU output),
// whose per-row maximum magnitude the producing GEMM has already reduced
// (rowmax, float bits): one thread per 16-byte lane slot of the bf16 layout
// (8 columns of one row), E4M3 of each value times 448 / max into the FP8
// layout; the thread holding columns 0..7 writes the row's scale.
__global__ __launch_bounds__(256) void quant_rows8_kernel(const uint16_t* __restrict__ a, int KB,
                                                          int M, int Mp, int RBm,
                                                          const uint32_t* __restrict__ rowmax,
                                                          uint8_t* __restrict__ a8,
                                                          float* __restrict__ sa) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int lane = (int)(gid & 63);
  const int64_t frag = gid >> 6;  // (kb, rb) over the row blocks that hold rows < M
  const int rb = (int)(frag % RBm), kb = (int)(frag / RBm);
  const int r = rb * 16 + (lane & 15), g = lane >> 4;
  if (kb >= KB || r >= M) return;
  const uint4 raw = *(const uint4*)(a + ((int64_t)(kb * (Mp >> 4) + rb) * 64 + lane) * 8);
  const float mx = __uint_as_float(rowmax[r]);
  const float si = e4m3_inv(mx);
  const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
  uint32_t b[2] = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    b[e >> 2] |= f32_to_e4m3(bf2f_bits((e & 1) ? w4[e >> 1] >> 16 : w4[e >> 1] & 0xffff) * si)
                 << (8 * (e & 3));
  *(uint2*)(a8 + packA8_off(r, kb * 32 + g * 8, Mp)) = make_uint2(b[0], b[1]);
  if (kb == 0 && g == 0) sa[r] = e4m3_scale(mx);
}

// Per source row of a bf16 weight [rows][K]: the FP8 scaling pair
// (inv = 448 / max|w|, scale = max|w| / 448). One workgroup per row.
__global__ __launch_bounds__(256) void rowscale_kernel(const uint16_t* __restrict__ w, int K,
                                                       float* __restrict__ inv,
                                                       float* __restrict__ scale) {
  __shared__ float redm[4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint16_t* wr = w + (int64_t)blockIdx.x * K;
  float mx = 0.f;
  for (int k = tid; k < K; k += 256) mx = fmaxf(mx, fabsf(bf2f_bits(wr[k])));
  mx = wave_max(mx);
  if (lane == 0) redm[wv] = mx;
  __syncthreads();
  if (tid == 0) {
    mx = fmaxf(fmaxf(redm[0], redm[1]), fmaxf(redm[2], redm[3]));
    inv[blockIdx.x] = e4m3_inv(mx);
    scale[blockIdx.x] = e4m3_scale(mx);
  }
}

// FP8 weight repack: the layout of repack_kernel with 16 E4M3 values (16
// bytes) per lane slot, i.e. unit (block, kk) of k-chunk kc holds columns
// kc 128 + kk 64 + 16 (lane / 16) .. + 15; the values are the bf16 weights
// times their row's inverse scale. sw gets the scale of every packed column
// (0 for padding columns). Up to three sources: concatenated rows, or (pairs)
// alternating blocks of the first two.
__global__ __launch_bounds__(256) void repack8_kernel(const uint16_t* __restrict__ s0,
                                                      const float* __restrict__ inv0,
                                                      const float* __restrict__ sc0, int r0,
                                                      const uint16_t* __restrict__ s1,
                                                      const float* __restrict__ inv1,
                                                      const float* __restrict__ sc1, int r1,
                                                      const uint16_t* __restrict__ s2,
                                                      const float* __restrict__ inv2,
                                                      const float* __restrict__ sc2, int r2,
                                                      int K, int KC, int NB, int64_t total,
                                                      int pairs, uint8_t* __restrict__ dst,
                                                      float* __restrict__ sw) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= total) return;
  const int lane = (int)(gid & 63);
  int64_t u = gid >> 6;
  const int kk = (int)(u & 1);
  u >>= 1;
  const int nbi = (int)(u % NB);
  u /= NB;
  const int kc = (int)(u % KC);
  const int blk = (int)(u / KC) * NB + nbi;
  const int k0 = kc * 128 + kk * 64 + (lane >> 4) * 16;
  const uint16_t* src = nullptr;
  float si = 0.f, sc = 0.f;
  int row = 0;
  if (pairs) {
    row = (blk >> 1) * 16 + (lane & 15);
    if (!(blk & 1)) { if (row < r0) { src = s0; si = inv0[row]; sc = sc0[row]; } }
    else { if (row < r1) { src = s1; si = inv1[row]; sc = sc1[row]; } }
  } else {
    const int n = blk * 16 + (lane & 15);
    if (n < r0) { src = s0; row = n; si = inv0[row]; sc = sc0[row]; }
    else if (n < r0 + r1) { src = s1; row = n - r0; si = inv1[row]; sc = sc1[row]; }
    else if (n < r0 + r1 + r2) { src = s2; row = n - r0 - r1; si = inv2[row]; sc = sc2[row]; }
  }
  uint32_t b[4] = {0u, 0u, 0u, 0u};
  if (src && k0 < K) {
    const uint4 h0 = *(const uint4*)(src + (int64_t)row * K + k0);
    const uint4 h1 = *(const uint4*)(src + (int64_t)row * K + k0 + 8);
    const uint32_t w8[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float v = bf2f_bits((e & 1) ? w8[e >> 1] >> 16 : w8[e >> 1] & 0xffff);
      b[e >> 2] |= f32_to_e4m3(v * si) << (8 * (e & 3));
    }
  }
  *(uint4*)(dst + gid * 16) = make_uint4(b[0], b[1], b[2], b[3]);
  if (kc == 0 && kk == 0 && (lane >> 4) == 0) sw[blk * 16 + (lane & 15)] = src ? sc : 0.f;
}

// (max, sum, argmax) state of a run of vocabulary tiles: sum of exp(logit -
// max); the lowest index among equal maxima
struct LmState {
  float m, s;
  int idx;
};
__device__ __forceinline__ LmState lm_combine(LmState a, LmState b) {
  const float nm = fmaxf(a.m, b.m);
  const float sa = a.m == -INFINITY ? 0.f : a.s * expf(a.m - nm);
  const float sb = b.m == -INFINITY ? 0.f : b.s * expf(b.m - nm);
  int ni;
  if (a.m > b.m) ni = a.idx;
  else if (b.m > a.m) ni = b.idx;
  else ni = a.idx < b.idx ? a.idx : b.idx;
  return {nm, sa + sb, ni};
}

// One workgroup per row: merge (max, sum, argmax) of all vocabulary tiles.
// Thread t takes tiles t, t + 256, ... (loads of four tiles in flight); the
// 256 states are then combined in a fixed tree (wavefront shuffles, then the
// four wavefronts in order), the same for every row.
__global__ __launch_bounds__(256) void lm_merge_kernel(const float* __restrict__ pm,
                                                       const float* __restrict__ ps,
                                                       const int32_t* __restrict__ pi, int M,
                                                       int tiles, float* __restrict__ conf,
                                                       int32_t* __restrict__ pred) {
  __shared__ LmState red[4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int r = blockIdx.x;
  LmState st{-INFINITY, 0.f, 0x7fffffff};
  const float* rm = pm + (int64_t)r * tiles;
  const float* rs = ps + (int64_t)r * tiles;
  const int32_t* ri = pi + (int64_t)r * tiles;
  // a thread's tiles tid, tid + 256, ... in order, LM_BATCH of them loaded
  // (index clamped, no load under a branch) before any is merged
  constexpr int LM_BATCH = 4;
  for (int t0 = tid; t0 < tiles; t0 += 256 * LM_BATCH) {
    float tm[LM_BATCH], ts[LM_BATCH];
    int ti[LM_BATCH];
#pragma unroll
    for (int b = 0; b < LM_BATCH; ++b) {
      const int t = min(t0 + 256 * b, tiles - 1);
      tm[b] = rm[t];
      ts[b] = rs[t];
      ti[b] = ri[t];
    }
#pragma unroll
    for (int b = 0; b < LM_BATCH; ++b)
      if (t0 + 256 * b < tiles && tm[b] != -INFINITY) st = lm_combine(st, {tm[b], ts[b], ti[b]});
  }
  for (int o = 1; o < 64; o <<= 1) {
    const LmState ot{__shfl_xor(st.m, o), __shfl_xor(st.s, o), __shfl_xor(st.idx, o)};
    st = lm_combine(st, ot);
  }
  if (lane == 0) red[wv] = st;
  __syncthreads();
  if (tid == 0) {
    st = lm_combine(lm_combine(red[0], red[1]), lm_combine(red[2], red[3]));
    conf[r] = 1.0f / st.s;
    pred[r] = (st.idx == 0x7fffffff) ? 0 : st.idx;  // all logits non-finite: report token 0
  }
}

// Weight repack: one thread per (fragment, lane) writes 8 bf16 (16 bytes);
// thread order is the packed order [tile][kc][block in tile][kk][lane].
__global__ __launch_bounds__(256) void repack_kernel(const uint16_t* __restrict__ s0, int r0,
                                                     const uint16_t* __restrict__ s1, int r1,
                                                     const uint16_t* __restrict__ s2, int r2,
                                                     int K, int KC, int NB, int64_t total,
                                                     int pairs, uint16_t* __restrict__ dst) {
  // K: length of a source row; KC * 64 >= K: packed columns, the excess is zero
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= total) return;
  const int lane = (int)(gid & 63);
  int64_t u = gid >> 6;
  const int kk = (int)(u & 1);
  u >>= 1;
  const int nbi = (int)(u % NB);
  u /= NB;
  const int kc = (int)(u % KC);
  const int blk = (int)(u / KC) * NB + nbi;
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
namespace {
// threads per row and 4-column groups per thread for a row of H columns:
// 1: (256, 1), 2: (512, 1), 3: (1024, 1), 4: (1024, 2)
int resnorm_shape(int H) { return H <= 1024 ? 1 : H <= 2048 ? 2 : H <= 4096 ? 3 : 4; }
}  // namespace

hipError_t launch_embed_norm(const int32_t* tokens, const uint16_t* embed, int vocab,
                             const float* w, float eps, int M, int Mp, int H, float* x,
                             uint16_t* a, hipStream_t s) {
  if (H % 256 || H > H_MAX) return hipErrorInvalidValue;
#define EMBEDNORM(NG, TPB)                                                                \
  hipLaunchKernelGGL((resnorm_kernel<true, 0, NG, false, TPB>), dim3(M), dim3(TPB), 0, s,      \
                     tokens, embed, vocab, nullptr, 0, w, eps, M, Mp, H, x, a, nullptr, nullptr, \
                     nullptr)
  switch (resnorm_shape(H)) {
    case 1: EMBEDNORM(1, 256); break;
    case 2: EMBEDNORM(1, 512); break;
    case 3: EMBEDNORM(1, 1024); break;
    default: EMBEDNORM(2, 1024); break;
  }
#undef EMBEDNORM
  return hipGetLastError();
}

hipError_t launch_embed_norm8(const int32_t* tokens, const uint16_t* embed, int vocab,
                              const float* w, float eps, int M, int Mp, int H, float* x,
                              uint8_t* a8, float* sa, uint32_t* rz, hipStream_t s) {
  if (H % 256 || H > H_MAX || !a8 || !sa) return hipErrorInvalidValue;
#define EMBEDNORM8(NG, TPB)                                                               \
  hipLaunchKernelGGL((resnorm_kernel<true, 0, NG, true, TPB>), dim3(M), dim3(TPB), 0, s,       \
                     tokens, embed, vocab, nullptr, 0, w, eps, M, Mp, H, x, nullptr, a8, sa, rz)
  switch (resnorm_shape(H)) {
    case 1: EMBEDNORM8(1, 256); break;
    case 2: EMBEDNORM8(1, 512); break;
    case 3: EMBEDNORM8(1, 1024); break;
    default: EMBEDNORM8(2, 1024); break;
  }
#undef EMBEDNORM8
  return hipGetLastError();
}

namespace {
template <int NG, bool A8, int TPB>
void resnorm_ng(const float* part, int S, const float* w, float eps, int M, int Mp, int H,
                float* x, uint16_t* a, uint8_t* a8, float* sa, uint32_t* rz, hipStream_t s) {
#define RESNORM(SC)                                                                         \
  hipLaunchKernelGGL((resnorm_kernel<false, SC, NG, A8, TPB>), dim3(M), dim3(TPB), 0, s, nullptr, \
                     nullptr, 0, part, S, w, eps, M, Mp, H, x, a, a8, sa, rz)
  switch (S) {
    case 0: RESNORM(0); break;
    case 2: RESNORM(2); break;
    case 3: RESNORM(3); break;
    case 4: RESNORM(4); break;
    case 5: RESNORM(5); break;
    case 6: RESNORM(6); break;
    case 7: RESNORM(7); break;
    case 8: RESNORM(8); break;
    case 9: RESNORM(9); break;
    default: RESNORM(-1); break;
  }
#undef RESNORM
}
}  // namespace

hipError_t launch_resnorm(const float* part, int S, const float* w, float eps, int M, int Mp,
                          int H, float* x, uint16_t* a, hipStream_t s) {
  if (H % 256 || H > H_MAX || S < 0) return hipErrorInvalidValue;
  switch (resnorm_shape(H)) {
    case 1: resnorm_ng<1, false, 256>(part, S, w, eps, M, Mp, H, x, a, nullptr, nullptr, nullptr, s); break;
    case 2: resnorm_ng<1, false, 512>(part, S, w, eps, M, Mp, H, x, a, nullptr, nullptr, nullptr, s); break;
    case 3: resnorm_ng<1, false, 1024>(part, S, w, eps, M, Mp, H, x, a, nullptr, nullptr, nullptr, s); break;
    default: resnorm_ng<2, false, 1024>(part, S, w, eps, M, Mp, H, x, a, nullptr, nullptr, nullptr, s); break;
  }
  return hipGetLastError();
}

hipError_t launch_resnorm8(const float* part, int S, const float* w, float eps, int M, int Mp,
                           int H, float* x, uint8_t* a8, float* sa, uint32_t* rz, hipStream_t s) {
  if (H % 256 || H > H_MAX || S < 0 || !a8 || !sa) return hipErrorInvalidValue;
  switch (resnorm_shape(H)) {
    case 1: resnorm_ng<1, true, 256>(part, S, w, eps, M, Mp, H, x, nullptr, a8, sa, rz, s); break;
    case 2: resnorm_ng<1, true, 512>(part, S, w, eps, M, Mp, H, x, nullptr, a8, sa, rz, s); break;
    case 3: resnorm_ng<1, true, 1024>(part, S, w, eps, M, Mp, H, x, nullptr, a8, sa, rz, s); break;
    default: resnorm_ng<2, true, 1024>(part, S, w, eps, M, Mp, H, x, nullptr, a8, sa, rz, s); break;
  }
  return hipGetLastError();
}

hipError_t launch_quant_rows8(const uint16_t* a, int K, int M, int Mp, const uint32_t* rowmax,
                              uint8_t* a8, float* sa, hipStream_t s) {
  if (K % 64 || M < 1 || M > Mp || !rowmax) return hipErrorInvalidValue;
  const int KB = K / 32, RBm = (M + 15) / 16;
  const int64_t threads = (int64_t)KB * RBm * 64;
  hipLaunchKernelGGL(quant_rows8_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     a, KB, M, Mp, RBm, rowmax, a8, sa);
  return hipGetLastError();
}

hipError_t launch_rowscale(const uint16_t* w, int rows, int K, float* inv, float* scale,
                           hipStream_t s) {
  hipLaunchKernelGGL(rowscale_kernel, dim3(rows), dim3(256), 0, s, w, K, inv, scale);
  return hipGetLastError();
}

hipError_t launch_repack8(const uint16_t* s0, const float* inv0, const float* sc0, int r0,
                          const uint16_t* s1, const float* inv1, const float* sc1, int r1,
                          const uint16_t* s2, const float* inv2, const float* sc2, int r2, int K,
                          int KP, int blocks, int nb, int pairs, uint8_t* dst, float* sw,
                          hipStream_t s) {
  if (KP % 512 || KP < K || K % 16 || nb < 1 || blocks % nb) return hipErrorInvalidValue;
  const int KC = KP / 128;
  const int64_t total = (int64_t)blocks * KC * 2 * 64;
  hipLaunchKernelGGL(repack8_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, s0,
                     inv0, sc0, r0, s1, inv1, sc1, r1, s2, inv2, sc2, r2, K, KC, nb, total, pairs,
                     dst, sw);
  return hipGetLastError();
}

hipError_t launch_lm_merge(const float* pm, const float* ps, const int32_t* pi, int M, int tiles,
                           float* conf, int32_t* pred, hipStream_t s) {
  hipLaunchKernelGGL(lm_merge_kernel, dim3(M), dim3(256), 0, s, pm, ps, pi, M, tiles, conf, pred);
  return hipGetLastError();
}

hipError_t launch_repack(const uint16_t* s0, int r0, const uint16_t* s1, int r1,
                         const uint16_t* s2, int r2, int K, int KP, int blocks, int nb, int pairs,
                         uint16_t* dst, hipStream_t s) {
  if (KP % 256 || KP < K || nb < 1 || blocks % nb) return hipErrorInvalidValue;
  const int KC = KP / 64;
  const int64_t total = (int64_t)blocks * KC * 2 * 64;
  const int64_t grid = (total + 255) / 256;
  hipLaunchKernelGGL(repack_kernel, dim3((unsigned)grid), dim3(256), 0, s, s0, r0, s1, r1, s2,
                     r2, K, KC, nb, total, pairs, dst);
  return hipGetLastError();
}


hipError_t launch_bf16_to_f32(const uint16_t* src, float* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

// bytes [0, n) of p set to zero, 16 bytes per thread (p and n multiples of 16)
__global__ __launch_bounds__(256) void fill_zero_kernel(uint4* p, int64_t n16) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) p[i] = make_uint4(0u, 0u, 0u, 0u);
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (((uintptr_t)p | bytes) & 15) return hipErrorInvalidValue;
  const int64_t n16 = (int64_t)(bytes / 16);
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, s,
                     (uint4*)p, n16);
  return hipGetLastError();
}

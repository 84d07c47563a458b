// Block attention of the verify forward (Sec. 3.3): every block row of branch b
// attends to all committed prefix positions [0, P) of the shared cache and to
// all L rows of its own branch (full attention inside the block); branches
// never see each other. Grouped-query: query head h reads KV head h / (Hq/Hkv).
//
// One workgroup per (query head, branch); one wavefront per 16 query rows.
// Scores are formed transposed, S^T = K Q^T, so that each lane owns one query
// row and the probabilities land directly in the operand layout of the
// second product O^T = V^T P^T (no cross-lane shuffle).
// Two passes over the keys: the first finds the exact row maximum, the second
// forms p = exp(s - max), rounds p to bf16 for the MFMA and accumulates the
// fp32 denominator. K tiles of 32 keys are staged in LDS, V tiles transposed.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

constexpr int KT = 32;  // keys per tile

template <int D>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int KP = D + 8;    // padded K row (bf16)
  constexpr int VP = KT + 8;   // padded V^T row (bf16)
  __shared__ __attribute__((aligned(16))) uint16_t sK[KT * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * VP];
  const int h = blockIdx.x, br = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nwaves = blockDim.x >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P, NK = P + L;
  const int row = wv * 16 + c16;  // this lane's query row inside the block
  const bool row_ok = row < L;

  // Q^T fragments: lane holds Q[row][32 kk + 8 g .. +8]
  uint4 qf[D / 32];
  const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * L + (row_ok ? row : 0)) * D;
  for (int kk = 0; kk < D / 32; ++kk)
    qf[kk] = row_ok ? *(const uint4*)(qrow + kk * 32 + g * 8) : make_uint4(0, 0, 0, 0);

  const uint16_t* kc = a.kcache + (int64_t)kvh * a.max_len * D;
  const uint16_t* vc = a.vcache + (int64_t)kvh * a.max_len * D;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + ((st_base + 0 * a.Hkv + kvh) * a.Lcap) * D;
  const uint16_t* vs = a.staging + ((st_base + 1 * a.Hkv + kvh) * a.Lcap) * D;
  const int ntiles = (NK + KT - 1) / KT;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  auto stage = [&](int t, bool with_v) {
    // KT keys x D dims, 8 dims (16 bytes) per item
    for (int q = tid; q < KT * (D / 8); q += blockDim.x) {
      const int kr = q / (D / 8), dg = q % (D / 8);
      const int key = t * KT + kr;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (key < P) {
        kv = *(const uint4*)(kc + (int64_t)key * D + dg * 8);
        if (with_v) vv = *(const uint4*)(vc + (int64_t)key * D + dg * 8);
      } else if (key < NK) {
        kv = *(const uint4*)(ks + (int64_t)(key - P) * D + dg * 8);
        if (with_v) vv = *(const uint4*)(vs + (int64_t)(key - P) * D + dg * 8);
      }
      *(uint4*)(sK + kr * KP + dg * 8) = kv;
      if (with_v) {
        const uint16_t* ve = (const uint16_t*)&vv;
        for (int e = 0; e < 8; ++e) sV[(dg * 8 + e) * VP + kr] = ve[e];
      }
    }
  };
  // S^T block for keys [t*KT + 16 kb, +16): acc[j] = s(key 16kb + 4g + j, row)
  auto scores = [&](int kb) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < D / 32; ++kk) {
      const uint4 kf = *(const uint4*)(sK + (kb * 16 + c16) * KP + kk * 32 + g * 8);
      s = mfma16(kf, qf[kk], s);
    }
    return s;
  };

  // pass 1: row maximum of the scaled scores
  float mx = -INFINITY;
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    stage(t, false);
    __syncthreads();
    for (int kb = 0; kb < 2; ++kb) {
      const f32x4 s = scores(kb);
      for (int j = 0; j < 4; ++j) {
        const int key = t * KT + kb * 16 + g * 4 + j;
        if (key < NK) mx = fmaxf(mx, s[j]);
      }
    }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));

  // pass 2: p = exp(s - max); O^T += V^T P^T
  f32x4 o[D / 16];
  for (int db = 0; db < D / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    stage(t, true);
    __syncthreads();
    uint16_t pb[8];
    for (int kb = 0; kb < 2; ++kb) {
      const f32x4 s = scores(kb);
      for (int j = 0; j < 4; ++j) {
        const int key = t * KT + kb * 16 + g * 4 + j;
        const float p = (key < NK) ? exp2f((s[j] - mx) * sl2) : 0.f;
        den += p;
        pb[kb * 4 + j] = f2bf_bits(p);
      }
    }
    const uint4 pf = *(const uint4*)pb;  // keys {4g+j} then {16+4g+j}
    for (int db = 0; db < D / 16; ++db) {
      const uint16_t* vr = sV + (db * 16 + c16) * VP;
      uint2 lo = *(const uint2*)(vr + g * 4), hi = *(const uint2*)(vr + 16 + g * 4);
      const uint4 vf = make_uint4(lo.x, lo.y, hi.x, hi.y);
      o[db] = mfma16(vf, pf, o[db]);  // o[db][j] = O^T(dim 16 db + 4g + j, row)
    }
  }
  den += __shfl_xor(den, 16);
  den += __shfl_xor(den, 32);
  if (!row_ok) return;
  const float inv = 1.0f / den;
  const int r = br * L + row;
  for (int db = 0; db < D / 16; ++db) {
    uint16_t ob[4];
    for (int j = 0; j < 4; ++j) ob[j] = f2bf_bits(o[db][j] * inv);
    const int col = h * D + db * 16 + g * 4;
    *(uint2*)(a.out + packA_off(r, col, a.Mp)) = *(const uint2*)ob;
  }
  (void)nwaves;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int waves = (a.L + 15) / 16;
  dim3 grid(a.Hq, a.nb), block(64 * waves);
  if (a.d == 128) hipLaunchKernelGGL(attn_kernel<128>, grid, block, 0, s, a);
  else if (a.d == 64) hipLaunchKernelGGL(attn_kernel<64>, grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

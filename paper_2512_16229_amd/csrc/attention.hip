// Block attention of the verify forward (Sec. 3.3): every block row of branch b
// attends to all committed prefix positions [0, P) of the shared cache and to
// all L rows of its own branch (full attention inside the block); branches
// never see each other. Grouped-query: query head h reads KV head h / (Hq/Hkv).
//
// One workgroup per (query head, branch) with four wavefronts; each wavefront
// takes a quarter of the key tiles (32 keys each) for all L rows, and the
// four partial softmax states are merged through LDS at the end. No K or V
// byte goes through LDS: both are read straight from global memory (L2) in
// MFMA operand layout. Scores are formed transposed, S^T = K Q^T, so a lane
// owns one query column and the probabilities land directly in the operand
// layout of O^T = V^T P^T; V is stored transposed ([d][position]) in the cache
// and the staging so that a lane's 8 keys of one dimension are two 8-byte runs.
// Prefix tiles and block tiles are kept apart (a tile reads one source, with
// positions aligned to 4) and keys past the end of either are masked: their
// probability and their V values are zero.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

constexpr int KT = 32;  // keys per tile

template <int D, int QB>
struct AttnTile {
  u32x4 k[2][D / 32];  // K fragments: key block kb, dims 32 kk + 8 g .. +8
  uint2 v[D / 16][2];  // V^T: dims 16 db + c16, keys {4g .. 4g+3} and {16 + 4g ..}
};

template <int D, int QB>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int NDB = D / 16, NKK = D / 32;
  __shared__ float sO[2][NDB * QB * 64 * 4];
  __shared__ float sM[2][QB * 16], sL[2][QB * 16];
  const int h = blockIdx.x, br = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P;
  const int pt = (P + KT - 1) / KT, bt = (L + KT - 1) / KT, T = pt + bt;
  const int t_lo = wv * T / 4, t_hi = (wv + 1) * T / 4;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  // Q^T operand: query column 16 qb + c16, dims 32 kk + 8 g .. +8
  u32x4 qf[QB][NKK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qb * 16 + c16;
    const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * L + (row < L ? row : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      qf[qb][kk] = row < L ? *(const u32x4*)(qrow + kk * 32 + g * 8) : u32x4{0u, 0u, 0u, 0u};
  }

  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;  // [pos][D]
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;  // [D][vld]
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;  // [pos][D]
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;  // [D][vlds]

  // tile t -> registers (positions past the end of the source read position 0)
  auto fetch = [&](int t, AttnTile<D, QB>& x) {
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT;  // first position of the tile in its source
    const int lim = pre ? P : L;
    const uint16_t* kb_ = pre ? kc : ks;
    const uint16_t* vb_ = pre ? vc : vs;
    const int64_t vld = pre ? a.vld : a.vlds;  // multiples of 8: a 4-key run stays in its row
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      int pos = p0 + kb * 16 + c16;
      pos = pos < lim ? pos : 0;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
        x.k[kb][kk] = *(const u32x4*)(kb_ + (int64_t)pos * D + kk * 32 + g * 8);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const uint16_t* vr = vb_ + (int64_t)(db * 16 + c16) * vld;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int pos = p0 + hf * 16 + g * 4;  // 4 keys pos .. pos + 3, 4-aligned
        x.v[db][hf] = pos < lim ? *(const uint2*)(vr + pos) : make_uint2(0u, 0u);
      }
    }
  };

  float m[QB], l[QB];  // running max (log2 units) and this lane's partial sum
  f32x4 o[NDB][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto compute = [&](int t, AttnTile<D, QB>& x) {
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT;
    const int lim = pre ? P : L;
    // zero V of masked keys (stale cache or staging contents may be non-finite)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int pos = p0 + hf * 16 + g * 4;
      if (pos + 3 >= lim) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          uint16_t* e = (uint16_t*)&x.v[db][hf];
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (pos + j >= lim) e[j] = 0;
        }
      }
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      f32x4 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) s[kb] = mfma16(x.k[kb][kk], qf[qb][kk], s[kb]);
      }
      // s[kb][j]: key p0 + 16 kb + 4 g + j, query 16 qb + c16
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pos = p0 + kb * 16 + g * 4 + j;
          s[kb][j] = pos < lim ? s[kb][j] * sl2 : -INFINITY;
          tmax = fmaxf(tmax, s[kb][j]);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float mn = fmaxf(m[qb], tmax);
      // a fully masked tile leaves mn = -inf: keep everything as it is
      const float alpha = mn == -INFINITY ? 1.f : exp2f(m[qb] - mn);
      m[qb] = mn;
      l[qb] *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db][qb] *= alpha;
      uint16_t pb[8];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = mn == -INFINITY ? 0.f : exp2f(s[kb][j] - mn);
          l[qb] += p;
          pb[kb * 4 + j] = f2bf_bits(p);
        }
      const u32x4 pf = *(const u32x4*)pb;  // keys {4g .. 4g+3} then {16 + 4g ..}
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const u32x4 vf = {x.v[db][0].x, x.v[db][0].y, x.v[db][1].x, x.v[db][1].y};
        o[db][qb] = mfma16(vf, pf, o[db][qb]);  // O^T(dim 16 db + 4g + j, query)
      }
    }
  };

  // two tiles in flight: x0 holds tile t, x1 tile t + 1
  AttnTile<D, QB> x0, x1;
  if (t_lo < t_hi) fetch(t_lo, x0);
  if (t_lo + 1 < t_hi) fetch(t_lo + 1, x1);
  for (int t = t_lo; t < t_hi; t += 2) {
    compute(t, x0);
    if (t + 2 < t_hi) fetch(t + 2, x0);
    if (t + 1 >= t_hi) break;
    compute(t + 1, x1);
    if (t + 3 < t_hi) fetch(t + 3, x1);
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    l[qb] += __shfl_xor(l[qb], 16);
    l[qb] += __shfl_xor(l[qb], 32);
  }

  // merge the four key ranges: (2, 3) into (0, 1), then 1 into 0
  auto put = [&](int slot) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        *(f32x4*)&sO[slot][((db * QB + qb) * 64 + lane) * 4] = o[db][qb];
    if (g == 0)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        sM[slot][qb * 16 + c16] = m[qb];
        sL[slot][qb * 16 + c16] = l[qb];
      }
  };
  auto take = [&](int slot) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float mo = sM[slot][qb * 16 + c16], lo = sL[slot][qb * 16 + c16];
      const float mn = fmaxf(m[qb], mo);
      const float fa = mn == -INFINITY ? 0.f : exp2f(m[qb] - mn);
      const float fb = mn == -INFINITY ? 0.f : exp2f(mo - mn);
      m[qb] = mn;
      l[qb] = l[qb] * fa + lo * fb;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        o[db][qb] = o[db][qb] * fa + *(const f32x4*)&sO[slot][((db * QB + qb) * 64 + lane) * 4] * fb;
    }
  };
  if (wv >= 2) put(wv - 2);
  __syncthreads();
  if (wv < 2) take(wv);
  __syncthreads();
  if (wv == 1) put(0);
  __syncthreads();
  if (wv != 0) return;
  take(0);

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qb * 16 + c16;
    if (row >= L) continue;
    const float inv = 1.0f / l[qb];
    const int r = br * L + row;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      uint16_t ob[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) ob[j] = f2bf_bits(o[db][qb][j] * inv);
      const int col = h * D + db * 16 + g * 4;
      *(uint2*)(a.out + packA_off(r, col, a.Mp)) = *(const uint2*)ob;
    }
  }
}

template <int D>
hipError_t launch_d(const AttnArgs& a, hipStream_t s) {
  const dim3 grid(a.Hq, a.nb);
  switch ((a.L + 15) / 16) {
    case 1: hipLaunchKernelGGL((attn_kernel<D, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_kernel<D, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((attn_kernel<D, 3>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((attn_kernel<D, 4>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.L < 1 || a.L > 64 || a.P < 0 || a.Hq % a.Hkv || a.vld % 8 || a.vlds % 8 ||
      a.L > a.vlds || a.P > a.vld)
    return hipErrorInvalidValue;
  if (a.d == 128) return launch_d<128>(a, s);
  if (a.d == 64) return launch_d<64>(a, s);
  return hipErrorInvalidValue;
}

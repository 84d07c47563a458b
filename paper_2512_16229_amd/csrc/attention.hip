// Block attention of the verify forward (Sec. 3.3): every block row of branch b
// attends to all committed prefix positions [0, P) of the shared cache and to
// all L rows of its own branch (full attention inside the block); branches
// never see each other. Grouped-query: query head h reads KV head h / (Hq/Hkv).
//
// One workgroup per (query head, branch); one wavefront per 16 query rows.
// Scores are formed transposed, S^T = K Q^T, so each lane owns one query row
// and the probabilities land directly in the operand layout of the second
// product O^T = V^T P^T (no cross-lane shuffle). One pass over the keys with a
// running row maximum (online softmax): p = exp(s - m_running) is rounded to
// bf16 for the MFMA; earlier partial sums are rescaled when the maximum grows.
// K tiles (row-major) and V tiles (transposed) of KT keys go through two LDS
// buffers; the next two tiles are in flight in registers meanwhile.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

template <int D, int KT, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void attn_kernel(AttnArgs a) {
  constexpr int NT = WAVES * 64;
  constexpr int KP = D + 8;    // padded K row (bf16)
  constexpr int VP = KT + 8;   // padded V^T row (bf16)
  constexpr int NI = KT * (D / 8) / NT;  // 16-byte items per thread per tensor per tile
  static_assert(NI * NT == KT * (D / 8), "tile must split evenly");
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][KT * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][D * VP];
  const int h = blockIdx.x, br = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P, NK = P + L;
  const int row = wv * 16 + c16;  // this lane's query row inside the block
  const bool row_ok = row < L;

  // Q^T fragments: lane holds Q[row][32 kk + 8 g .. +8]
  u32x4 qf[D / 32];
  const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * L + (row_ok ? row : 0)) * D;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk)
    qf[kk] = row_ok ? *(const u32x4*)(qrow + kk * 32 + g * 8) : u32x4{0u, 0u, 0u, 0u};

  const uint16_t* kc = a.kcache + (int64_t)kvh * a.max_len * D;
  const uint16_t* vc = a.vcache + (int64_t)kvh * a.max_len * D;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + ((st_base + 0 * a.Hkv + kvh) * a.Lcap) * D;
  const uint16_t* vs = a.staging + ((st_base + 1 * a.Hkv + kvh) * a.Lcap) * D;
  const int ntiles = (NK + KT - 1) / KT;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  // tile t -> registers: item q = tid + i * NT covers key q / (D/8), dims 8 * (q % (D/8))
  auto fetch = [&](int t, u32x4 (&kr)[NI], u32x4 (&vr)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = tid + i * NT;
      const int key = t * KT + q / (D / 8), dg = q % (D / 8);
      u32x4 k4 = {0u, 0u, 0u, 0u}, v4 = {0u, 0u, 0u, 0u};
      if (key < P) {
        k4 = *(const u32x4*)(kc + (int64_t)key * D + dg * 8);
        v4 = *(const u32x4*)(vc + (int64_t)key * D + dg * 8);
      } else if (key < NK) {
        k4 = *(const u32x4*)(ks + (int64_t)(key - P) * D + dg * 8);
        v4 = *(const u32x4*)(vs + (int64_t)(key - P) * D + dg * 8);
      }
      kr[i] = k4;
      vr[i] = v4;
    }
  };
  auto stash = [&](int buf, const u32x4 (&kr)[NI], const u32x4 (&vr)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = tid + i * NT;
      const int kr_ = q / (D / 8), dg = q % (D / 8);
      *(u32x4*)(&sK[buf][kr_ * KP + dg * 8]) = kr[i];
      const uint16_t* ve = (const uint16_t*)&vr[i];
#pragma unroll
      for (int e = 0; e < 8; ++e) sV[buf][(dg * 8 + e) * VP + kr_] = ve[e];
    }
  };

  float m = -INFINITY, den = 0.f;  // running max (log2 units) and this lane's partial sum
  f32x4 o[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int t, int buf) {
    f32x4 s[KT / 16];
#pragma unroll
    for (int kb = 0; kb < KT / 16; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        const u32x4 kf = *(const u32x4*)(&sK[buf][(kb * 16 + c16) * KP + kk * 32 + g * 8]);
        s[kb] = mfma16(kf, qf[kk], s[kb]);
      }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < KT / 16; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = t * KT + kb * 16 + g * 4 + j;
        s[kb][j] = (key < NK) ? s[kb][j] * sl2 : -INFINITY;
        tmax = fmaxf(tmax, s[kb][j]);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mn = fmaxf(m, tmax);
    const float alpha = exp2f(m - mn);  // 0 on the first tile (m = -inf)
    m = mn;
    den *= alpha;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) o[db] *= alpha;
#pragma unroll
    for (int c = 0; c < KT / 32; ++c) {
      uint16_t pb[8];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = exp2f(s[2 * c + hh][j] - mn);  // exp2(-inf) = 0 for masked keys
          den += p;
          pb[hh * 4 + j] = f2bf_bits(p);
        }
      const u32x4 pf = *(const u32x4*)pb;  // keys {32c + 4g + j} then {32c + 16 + 4g + j}
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        const uint16_t* vr = &sV[buf][(db * 16 + c16) * VP + c * 32];
        const uint2 lo = *(const uint2*)(vr + g * 4), hi = *(const uint2*)(vr + 16 + g * 4);
        const u32x4 vf = {lo.x, lo.y, hi.x, hi.y};
        o[db] = mfma16(vf, pf, o[db]);  // o[db][j] = O^T(dim 16 db + 4g + j, row)
      }
    }
  };

  u32x4 k0[NI], v0[NI], k1[NI], v1[NI];
  fetch(0, k0, v0);
  if (ntiles > 1) fetch(1, k1, v1);
  stash(0, k0, v0);
  if (ntiles > 2) fetch(2, k0, v0);
  for (int t = 0; t < ntiles; t += 2) {
    // tile t in LDS buffer 0; t+1 in registers k1/v1; t+2 in flight into k0/v0
    lds_barrier();
    if (t + 1 < ntiles) stash(1, k1, v1);
    if (t + 3 < ntiles) fetch(t + 3, k1, v1);
    compute(t, 0);
    if (t + 1 >= ntiles) break;
    lds_barrier();
    if (t + 2 < ntiles) stash(0, k0, v0);
    if (t + 4 < ntiles) fetch(t + 4, k0, v0);
    compute(t + 1, 1);
  }
  den += __shfl_xor(den, 16);
  den += __shfl_xor(den, 32);
  if (!row_ok) return;
  const float inv = 1.0f / den;
  const int r = br * L + row;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    uint16_t ob[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) ob[j] = f2bf_bits(o[db][j] * inv);
    const int col = h * D + db * 16 + g * 4;
    *(uint2*)(a.out + packA_off(r, col, a.Mp)) = *(const uint2*)ob;
  }
}

template <int D>
hipError_t launch_d(const AttnArgs& a, hipStream_t s) {
  const int waves = (a.L + 15) / 16;
  const dim3 grid(a.Hq, a.nb);
  switch (waves) {
    case 1: hipLaunchKernelGGL((attn_kernel<D, 32, 1>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_kernel<D, 64, 2>), grid, dim3(128), 0, s, a); break;
    case 3:
    case 4: hipLaunchKernelGGL((attn_kernel<D, 64, 4>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.d == 128) return launch_d<128>(a, s);
  if (a.d == 64) return launch_d<64>(a, s);
  return hipErrorInvalidValue;
}

// Block attention of the verify forward (Sec. 3.3): every block row of branch b
// attends to all committed prefix positions [0, P) of the shared cache and to
// all L rows of its own branch (full attention inside the block); branches
// never see each other. Grouped-query: query head h reads KV head h / (Hq/Hkv).
//
// One workgroup per (query head, branch) with four wavefronts; each wavefront
// takes a quarter of the key tiles (32 keys each) for all L rows, and the
// four partial softmax states are merged through LDS at the end. Each
// wavefront streams its tiles through a private two-slot LDS ring with
// asynchronous global -> LDS copies (one tile in flight while the previous one
// is computed), then reads the K and V fragments from LDS in MFMA operand
// layout. Scores are formed transposed, S^T = K Q^T, so a lane owns one query
// column and the probabilities land directly in the operand layout of
// O^T = V^T P^T; V is stored transposed ([d][position]) in the cache and the
// staging so that a copy lane's 8 keys of one dimension are 16 contiguous bytes.
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

// Asynchronous copy of 16 bytes per lane, from base + voff(lane) (base
// wave-uniform, in SGPRs) to bytes [16 lane, 16 lane + 16) of the 1 KiB LDS
// block at lds_addr (wave-uniform, in M0). The compiler does not track it:
// completion is awaited with an explicit vmcnt wait.
__device__ __forceinline__ void attn_dma16(const void* base, uint32_t voff, uint32_t lds_addr) {
  const uint64_t u = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  const void* sbase = (const void*)(((uint64_t)hi << 32) | lo);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               ::"s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(sbase)
               : "memory");
}
// max / sum of the values of lanes l and l ^ 16 (l ^ 32): the permlane swaps
// hand each lane both values of its pair, lower lane first, so the two lanes
// of a pair get bitwise identical results
__device__ __forceinline__ float pair16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair16_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int N>
__device__ __forceinline__ void attn_wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int D, int QB>
struct AttnSmem {
  static constexpr int NDB = D / 16, NKK = D / 32;
  static constexpr int KBYTES = 2 * NKK * 1024;   // K of one tile: [kb][kk][lane][16 B]
  static constexpr int TILE = KBYTES + NDB * 1024;  // + V^T: [db][lane][16 B]
  static constexpr int RING = 4 * 2 * TILE;         // four wavefronts x two slots
  static constexpr int MERGE_O = NDB * QB * 64 * 4;  // floats of one merge slot
  static constexpr int MERGE = (2 * MERGE_O + 4 * QB * 16) * 4;
  static constexpr int BYTES = RING > MERGE ? RING : MERGE;
  static constexpr int OPS = 2 * NKK + NDB;  // copies per tile and wavefront
};

template <int D, int QB>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  using SM = AttnSmem<D, QB>;
  constexpr int NDB = D / 16, NKK = D / 32;
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];
  const int h = blockIdx.x, br = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P;
  const int pt = (P + KT - 1) / KT, bt = (L + KT - 1) / KT, T = pt + bt;
  const int t_lo = wv * T / 4, t_hi = (wv + 1) * T / 4;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;  // [pos][D]
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;  // [D][vld]
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;  // [pos][D]
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;  // [D][vlds]
  const uint32_t ring = (uint32_t)(uintptr_t)smem + (uint32_t)(wv * 2) * SM::TILE;

  // tile t -> ring slot: OPS copies, each from a wave-uniform base at the
  // tile's first position plus a per-lane byte offset. A K copy lane takes key
  // row 16 kb + c16, dims 32 kk + 8 g .. +8; a V copy lane dimension
  // 16 db + c16, keys 8 g .. 8 g + 7. In a tile that runs past the end of its
  // source, K rows past the end read the last row and V runs that start past
  // the end read the first run (compute() masks both): every copy stays inside
  // the source, whose row lengths are multiples of 8.
  const uint32_t koff_full[2] = {(uint32_t)((c16 * D + g * 8) * 2),
                                 (uint32_t)(((16 + c16) * D + g * 8) * 2)};
  const uint32_t voff_pre = (uint32_t)((c16 * a.vld + 8 * g) * 2);
  const uint32_t voff_blk = (uint32_t)((c16 * a.vlds + 8 * g) * 2);
  auto issue = [&](int t, int slot) {
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT;
    const int lim = pre ? P : L;
    const int64_t vld = pre ? a.vld : a.vlds;
    const uint16_t* kb_ = (pre ? kc : ks) + (int64_t)p0 * D;
    const uint16_t* vb_ = (pre ? vc : vs) + p0;
    uint32_t koff[2] = {koff_full[0], koff_full[1]};
    uint32_t voff = pre ? voff_pre : voff_blk;
    if (p0 + KT > lim) {  // wave-uniform: the last, partial tile of a source
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int r = kb * 16 + c16 < lim - p0 ? kb * 16 + c16 : lim - 1 - p0;
        koff[kb] = (uint32_t)((r * D + g * 8) * 2);
      }
      voff = (uint32_t)((c16 * vld + (8 * g < lim - p0 ? 8 * g : 0)) * 2);
    }
    const uint32_t sb = ring + (uint32_t)slot * SM::TILE;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) attn_dma16(kb_ + kk * 32, koff[kb], sb + (kb * NKK + kk) * 1024);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      attn_dma16(vb_ + (int64_t)db * 16 * vld, voff, sb + SM::KBYTES + db * 1024);
  };

  // ring slot -> registers (operand layouts)
  auto fetch = [&](int slot, AttnTile<D, QB>& x) {
    const char* sb = smem + (wv * 2 + slot) * SM::TILE;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
        x.k[kb][kk] = *(const u32x4*)(sb + ((kb * NKK + kk) * 64 + lane) * 16);
    // keys 4g .. 4g+3 sit in copy lane c16 + 16 (g / 2) at byte 8 (g % 2);
    // keys 16 + 4g .. in copy lane c16 + 16 (2 + g / 2)
    const char* vb = sb + SM::KBYTES + (c16 + 16 * (g >> 1)) * 16 + 8 * (g & 1);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      x.v[db][0] = *(const uint2*)(vb + db * 1024);
      x.v[db][1] = *(const uint2*)(vb + db * 1024 + 32 * 16);
    }
  };

  // the first two tiles are in flight while Q is loaded
  const int n = t_hi - t_lo;
  if (n > 0) {
    issue(t_lo, 0);
    issue(t_lo + (n > 1 ? 1 : 0), 1);
  }

  // Q^T operand: query column 16 qb + c16, dims 32 kk + 8 g .. +8
  u32x4 qf[QB][NKK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qb * 16 + c16;
    const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * L + (row < L ? row : 0)) * D;
    const unsigned keep = row < L ? ~0u : 0u;  // rows past L: zero queries
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[qb][kk] = *(const u32x4*)(qrow + kk * 32 + g * 8) & keep;
  }

  float m[QB], l[QB];  // running max (log2 units) and this lane's partial sum
  f32x4 o[NDB][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // One key tile for all query rows. The probabilities are taken against a
  // reference maximum m that trails the running row maximum by at most 8
  // (log2 units): m, l and o are rescaled only when some row's maximum has
  // grown past that (a wave-uniform decision), so p = 2^(s - m) <= 2^8.
  // o / l and the final merge are unchanged by the choice of reference.
  auto compute = [&](int t, AttnTile<D, QB>& x) {
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT;
    const int lim = pre ? P : L;
    const bool full = p0 + KT <= lim;  // wave-uniform
    if (!full) {
      // zero V of masked keys (stale cache or staging contents may be
      // non-finite, and 0 * inf would poison the sums)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int pos = p0 + hf * 16 + g * 4;
        const unsigned m01 = (pos < lim ? 0xFFFFu : 0u) | (pos + 1 < lim ? 0xFFFF0000u : 0u);
        const unsigned m23 = (pos + 2 < lim ? 0xFFFFu : 0u) | (pos + 3 < lim ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          x.v[db][hf].x &= m01;
          x.v[db][hf].y &= m23;
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
      if (full) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) s[kb] *= sl2;
      } else {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int pos = p0 + kb * 16 + g * 4 + j;
            s[kb][j] = pos < lim ? s[kb][j] * sl2 : -INFINITY;
          }
      }
      float tmax = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
      tmax = pair32_max(pair16_max(tmax));
      const float mn = fmaxf(m[qb], tmax);
      if (__builtin_amdgcn_ballot_w64(mn > m[qb] + 8.f)) {
        // m = -inf (nothing seen yet) gives alpha = 0 on zero o and l
        const float alpha = mn == -INFINITY ? 1.f : exp2f(m[qb] - mn);
        m[qb] = mn;
        l[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[db][qb] *= alpha;
      }
      const float mr = m[qb];
      uint16_t pb[8];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = mr == -INFINITY ? 0.f : exp2f(s[kb][j] - mr);
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

  // tile i sits in slot i % 2. At the top of an iteration tiles i and i + 1
  // are in flight (2 OPS copies): wait for the older one, compute it, and
  // refill its slot with tile i + 2 once its LDS reads have completed. Past
  // the last tile the last one is copied again (an L2 hit), so the number of
  // copies in flight is the same in every iteration.
  for (int i = 0; i < n; ++i) {
    attn_wait_vmcnt<SM::OPS>();
    AttnTile<D, QB> x;
    fetch(i & 1, x);
    compute(t_lo + i, x);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    issue(t_lo + (i + 2 < n ? i + 2 : n - 1), i & 1);
  }
  attn_wait_vmcnt<0>();  // the ring is reused for the merge
  __syncthreads();
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    l[qb] = pair32_sum(pair16_sum(l[qb]));
  }

  // merge the four key ranges: (2, 3) into (0, 1), then 1 into 0
  float(*sO)[SM::MERGE_O] = (float(*)[SM::MERGE_O])smem;
  float(*sM)[QB * 16] = (float(*)[QB * 16])(smem + 2 * SM::MERGE_O * 4);
  float(*sL)[QB * 16] = (float(*)[QB * 16])(smem + 2 * SM::MERGE_O * 4 + 2 * QB * 16 * 4);
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

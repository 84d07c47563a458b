// Block attention of the verify forward (Sec. 3.3): every block row of branch b
// attends to all committed prefix positions [0, P) of the shared cache and to
// all L rows of its own branch (full attention inside the block); branches
// never see each other. Grouped-query: query head h reads KV head h / (Hq/Hkv).
//
// One workgroup per (query head, branch) with four wavefronts; each wavefront
// takes a quarter of the key tiles (32 keys each, prefix tiles from the cache
// and block tiles from the branch's staging) for all L rows. The prefix K/V
// are read from HBM once per KV head per layer (the workgroups of a KV head
// find them in L2). The softmax takes two passes over the tiles: pass 1 forms
// the scores and each row's largest score (over the four wavefronts, through
// LDS); pass 2 forms them again (the same instructions, the same bits) and
// rounds each probability to bf16 against that exact maximum before it meets
// V, so no state is rescaled and the four partial states add up.
// K and V live in the KV tile layout (common.h): every 1 KiB MFMA operand
// fragment of a 32-key tile is one contiguous run, so tiles go global -> LDS
// (or straight into registers) by fully coalesced 16-byte lane copies, and a
// lane's scores S^T = K Q^T come out as keys 8 g .. 8 g + 7 of the tile for
// query c16, the order in which the probabilities meet V in O^T = V^T P^T.
// Keys past the end of a source (the last prefix tile, a block shorter than
// 32) are masked: their scores are -inf and their V values zero.
#include "common.h"
#include "kernels.h"

#include <math.h>

#include <algorithm>
#include <type_traits>

namespace {

constexpr int KT = 32;  // keys per tile

template <int D>
struct AttnTile {
  u32x4 k[2][D / 32];  // K fragments (kb, kk) in the KV tile layout
  u32x4 v[D / 16];     // V^T: dims 16 db + c16, keys 8 g .. 8 g + 7
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
// Maximum of scores (never NaN: finite bf16 products or the -inf of a masked
// key). This file is compiled without NaN semantics, so fmaxf maps to the
// hardware maximum without first quieting each operand.
__device__ __forceinline__ float max2(float a, float b) { return fmaxf(a, b); }
__device__ __forceinline__ float max3(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }
// max / sum of the values of lanes l and l ^ 16 (l ^ 32): the permlane swaps
// hand each lane both values of its pair, lower lane first, so the two lanes
// of a pair get bitwise identical results
__device__ __forceinline__ float pair16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair16_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// 2^x by the hardware instruction (no scaling of results below the normal
// range: such probabilities are < 2^-126 of the row maximum and flush to 0)
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }


template <int N>
__device__ __forceinline__ void attn_wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int D>
struct TileLds {
  static constexpr int NDB = D / 16, NKK = D / 32;
  static constexpr int KBYTES = 2 * NKK * 1024;     // K of one tile: [kb][kk][lane][16 B]
  static constexpr int TILE = KBYTES + NDB * 1024;  // + V^T: [db][lane][16 B]
  static constexpr int OPS = 2 * NKK + NDB;         // 1 KiB copies per tile
};

// Copy q (0 <= q < OPS) of the tile whose K and V (KV tile layout) start at
// kt and vt into the LDS slot at sb: K fragment q, or V fragment q - 2 D/32;
// each a contiguous 1 KiB, lane l taking bytes [16 l, 16 l + 16).
template <int D>
__device__ __forceinline__ void tile_copy(int q, const uint16_t* kt, const uint16_t* vt,
                                          uint32_t sb, int lane) {
  using T = TileLds<D>;
  const uint16_t* src = q < 2 * T::NKK ? kt + q * 512 : vt + (q - 2 * T::NKK) * 512;
  attn_dma16(src, (uint32_t)lane * 16u, sb + q * 1024);
}

// LDS slot -> registers (operand layouts)
template <int D>
__device__ __forceinline__ void tile_fetch(const char* sb, int lane, AttnTile<D>& x) {
  using T = TileLds<D>;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int kk = 0; kk < T::NKK; ++kk)
      x.k[kb][kk] = *(const u32x4*)(sb + ((kb * T::NKK + kk) * 64 + lane) * 16);
#pragma unroll
  for (int db = 0; db < T::NDB; ++db)
    x.v[db] = *(const u32x4*)(sb + T::KBYTES + (db * 64 + lane) * 16);
}

// Pass 2 of one key tile (keys p0 .. p0 + 31 of a source of lim positions) for
// NR blocks of 16 query rows; ALWAYS_FULL: the caller knows the tile lies
// wholly inside the source (no masking code). With s the raw score q.k and
// sl2 = scale log2(e), p = 2^(s sl2 - m) against the row's exact maximum m
// (log2 units, from pass 1), so p <= 1 and no state is ever rescaled; l sums
// the unrounded p, and V meets p rounded to bf16.
template <int D, int NR, bool ALWAYS_FULL>
__device__ __forceinline__ void tile_update(AttnTile<D>& x, const u32x4 (&qf)[NR][D / 32],
                                            const float (&m)[NR], float (&l)[NR],
                                            f32x4 (&o)[D / 16][NR], int p0, int lim, float sl2,
                                            int g, int cblk = 0, int row0 = 0) {
  constexpr int NDB = D / 16, NKK = D / 32;
  const bool full = ALWAYS_FULL || p0 + KT <= lim;  // wave-uniform
  if (!full) {
    // zero V of masked keys (stale cache or staging contents may be
    // non-finite, and 0 * inf would poison the sums); branch-free
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int pos = p0 + 8 * g + 2 * e;
      const unsigned mk = (pos < lim ? 0xFFFFu : 0u) | (pos + 1 < lim ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int db = 0; db < NDB; ++db) x.v[db][e] &= mk;
    }
  }
#pragma unroll
  for (int qb = 0; qb < NR; ++qb) {
    // block-causal mask (cblk > 0, a multiple of 16): rows row0 + 16 qb .. lie
    // in one sub-block and see the keys of the sub-blocks up to their own
    int lq = lim;
    if (cblk) {
      lq = min(lim, ((row0 + qb * 16) / cblk + 1) * cblk);
      if (p0 >= lq) continue;  // no key of this tile is visible to these rows
    }
    f32x4 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) s[kb] = mfma16(x.k[kb][kk], qf[qb][kk], s[kb]);
    }
    // s[kb][j]: key p0 + 8 g + 4 kb + j, query 16 qb + c16
    if (!full || p0 + KT > lq) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pos = p0 + 8 * g + 4 * kb + j;
          s[kb][j] = pos < lq ? s[kb][j] : -INFINITY;
        }
    }
    const float nm = -m[qb];
    uint16_t pb[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p = fast_exp2(__builtin_fmaf(s[kb][j], sl2, nm));  // masked: 2^-inf = 0
        l[qb] += p;
        pb[kb * 4 + j] = f2bf_bits(p);
      }
    const u32x4 pf = *(const u32x4*)pb;  // keys 8 g .. 8 g + 7
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      o[db][qb] = mfma16(x.v[db], pf, o[db][qb]);  // O^T(dim 16 db + 4g + j, query)
  }
}

// Pass 1 of the two-pass softmax: the largest raw score q.k of each query
// column over the keys of one tile (K fragments read from the LDS slot sb),
// with the same masking as tile_update; mraw keeps the running maximum.
template <int D, int NR>
__device__ __forceinline__ void tile_max(const char* sb, int lane, const u32x4 (&qf)[NR][D / 32],
                                         float (&mraw)[NR], int p0, int lim, int g, int cblk,
                                         int row0) {
  constexpr int NKK = D / 32;
  u32x4 kf[2][NKK];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      kf[kb][kk] = *(const u32x4*)(sb + ((kb * NKK + kk) * 64 + lane) * 16);
#pragma unroll
  for (int qb = 0; qb < NR; ++qb) {
    int lq = lim;
    if (cblk) {
      lq = min(lim, ((row0 + qb * 16) / cblk + 1) * cblk);
      if (p0 >= lq) continue;
    }
    f32x4 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) s[kb] = mfma16(kf[kb][kk], qf[qb][kk], s[kb]);
    }
    if (p0 + KT > lq) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pos = p0 + 8 * g + 4 * kb + j;
          s[kb][j] = pos < lq ? s[kb][j] : -INFINITY;
        }
    }
    mraw[qb] = max2(mraw[qb], max2(max3(s[0][0], s[0][1], s[0][2]),
                                   max3(max3(s[0][3], s[1][0], s[1][1]), s[1][2], s[1][3])));
  }
}

template <int D, int QB>
struct AttnSmem {
  static constexpr int NDB = D / 16;
  static constexpr int RING = 4 * 2 * TileLds<D>::TILE;  // four wavefronts x two slots
  static constexpr int MERGE_O = NDB * QB * 64 * 4;      // floats of one merge slot
  static constexpr int MERGE = (2 * MERGE_O + 2 * QB * 16) * 4;
  static constexpr int BYTES = RING > MERGE ? RING : MERGE;
  static constexpr int OPS = TileLds<D>::OPS;
};

// Per (query head, branch): the prefix tiles and the block tiles.
template <int D, int QB>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  using SM = AttnSmem<D, QB>;
  constexpr int NDB = D / 16, NKK = D / 32;
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];
  const int h = blockIdx.x, br = blockIdx.y;
  const int row0 = blockIdx.z * QB * 16;  // first query row of this workgroup's group
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P;
  const int pt = (P + KT - 1) / KT, bt = (L + KT - 1) / KT, T = pt + bt;
  const int t_lo = wv * T / 4, t_hi = (wv + 1) * T / 4;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;  // KV tile layout
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;
  const uint32_t ring = (uint32_t)(uintptr_t)smem + (uint32_t)(wv * 2) * TileLds<D>::TILE;

  // tile t -> this wavefront's ring slot: all OPS copies, or the K copies only
  // (pass 1); tiles are whole in memory (positions past the source are masked)
  auto issue = [&](int t, int slot) {
    const bool pre = t < pt;
    const int64_t off = (int64_t)(pre ? t : t - pt) * KT * D;
    const uint32_t sb = ring + (uint32_t)slot * TileLds<D>::TILE;
#pragma unroll
    for (int q = 0; q < SM::OPS; ++q) tile_copy<D>(q, (pre ? kc : ks) + off, (pre ? vc : vs) + off, sb, lane);
  };
  auto issue_k = [&](int t, int slot) {
    const bool pre = t < pt;
    const int64_t off = (int64_t)(pre ? t : t - pt) * KT * D;
    const uint32_t sb = ring + (uint32_t)slot * TileLds<D>::TILE;
#pragma unroll
    for (int q = 0; q < 2 * NKK; ++q) tile_copy<D>(q, (pre ? kc : ks) + off, (pre ? vc : vs) + off, sb, lane);
  };

  // the first two tiles are in flight while Q is loaded. The query heads of
  // one KV head start at different tiles of the range (and wrap), so that
  // their workgroups do not request the same K/V lines at the same moment.
  const int n = t_hi - t_lo;
  const int rot = n > 0 ? (h % (a.Hq / a.Hkv)) % n : 0;
  auto tile_of = [&](int i) { const int r = i + rot; return t_lo + (r < n ? r : r - n); };
  if (n > 0) {
    issue_k(tile_of(0), 0);
    issue_k(tile_of(n > 1 ? 1 : 0), 1);
  }

  // Q^T operand: query column 16 qb + c16, dims 32 kk + 8 g .. +8
  u32x4 qf[QB][NKK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = row0 + qb * 16 + c16;
    const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * L + (row < L ? row : 0)) * D;
    const unsigned keep = row < L ? ~0u : 0u;  // rows past L: zero queries
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[qb][kk] = *(const u32x4*)(qrow + kk * 32 + g * 8) & keep;
  }

  // Pass 1: each row's largest score over this wavefront's tiles (K only,
  // the same ring and order), then over the four wavefronts: the exact row
  // maximum, against which pass 2 rounds every probability.
  float mraw[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) mraw[qb] = -INFINITY;
  for (int i = 0; i < n; ++i) {
    attn_wait_vmcnt<2 * NKK>();
    const int t = tile_of(i);
    const bool pre = t < pt;
    tile_max<D, QB>(smem + (wv * 2 + (i & 1)) * TileLds<D>::TILE, lane, qf, mraw,
                    (pre ? t : t - pt) * KT, pre ? P : L, g, pre ? 0 : a.cblk, row0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    issue_k(tile_of(i + 2 < n ? i + 2 : n - 1), i & 1);
  }
  attn_wait_vmcnt<0>();
  __shared__ float s_max[4][QB * 16];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    mraw[qb] = pair32_max(pair16_max(mraw[qb]));
    if (g == 0) s_max[wv][qb * 16 + c16] = mraw[qb];
  }
  __syncthreads();
  float m[QB], l[QB];  // reference max (log2 units) and this lane's partial sum
  f32x4 o[NDB][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float mx = max2(max2(s_max[0][qb * 16 + c16], s_max[1][qb * 16 + c16]),
                          max2(s_max[2][qb * 16 + c16], s_max[3][qb * 16 + c16]));
    m[qb] = mx * sl2;  // every probability 2^(s sl2 - m) <= 1: never rescaled
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // Pass 2: the first two tiles again, K and V
  if (n > 0) {
    issue(tile_of(0), 0);
    issue(tile_of(n > 1 ? 1 : 0), 1);
  }

  // tile i sits in slot i % 2. At the top of an iteration tiles i and i + 1
  // are in flight (2 OPS copies): wait for the older one, compute it, and
  // refill its slot with tile i + 2 once its LDS reads have completed. Past
  // the last tile the last one is copied again (an L2 hit), so the number of
  // copies in flight is the same in every iteration.
  for (int i = 0; i < n; ++i) {
    attn_wait_vmcnt<SM::OPS>();
    AttnTile<D> x;
    tile_fetch<D>(smem + (wv * 2 + (i & 1)) * TileLds<D>::TILE, lane, x);
    const int t = tile_of(i);
    const bool pre = t < pt;
    tile_update<D, QB, false>(x, qf, m, l, o, (pre ? t : t - pt) * KT, pre ? P : L, sl2, g,
                              pre ? 0 : a.cblk, row0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    issue(tile_of(i + 2 < n ? i + 2 : n - 1), i & 1);
  }
  attn_wait_vmcnt<0>();  // the ring is reused for the merge
  __syncthreads();
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) l[qb] = pair32_sum(pair16_sum(l[qb]));

  // the four key ranges share the reference maximum: their states add up,
  // (2, 3) into (0, 1), then 1 into 0 (a fixed order)
  float(*sO)[SM::MERGE_O] = (float(*)[SM::MERGE_O])smem;
  float(*sL)[QB * 16] = (float(*)[QB * 16])(smem + 2 * SM::MERGE_O * 4);
  auto put = [&](int slot) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        *(f32x4*)&sO[slot][((db * QB + qb) * 64 + lane) * 4] = o[db][qb];
    if (g == 0)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sL[slot][qb * 16 + c16] = l[qb];
  };
  auto take = [&](int slot) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      l[qb] += sL[slot][qb * 16 + c16];
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        o[db][qb] += *(const f32x4*)&sO[slot][((db * QB + qb) * 64 + lane) * 4];
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
    const int row = row0 + qb * 16 + c16;
    const bool ok = row < L;
    const float inv = ok ? 1.0f / l[qb] : 0.f;
    const int r = br * L + row;
    float mrow = 0.f;  // largest |stored value| of this lane's part of the row
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      uint16_t ob[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ob[j] = f2bf_bits(o[db][qb][j] * inv);
        mrow = fmaxf(mrow, fabsf(bf2f_bits(ob[j])));
      }
      const int col = h * D + db * 16 + g * 4;
      if (ok) *(uint2*)(a.out + packA_off(r, col, a.Mp)) = *(const uint2*)ob;
    }
    if (a.rowmax) {  // lanes c16 + 16 g hold the row's 4 column groups of this head
      mrow = fmaxf(mrow, __shfl_xor(mrow, 16));
      mrow = fmaxf(mrow, __shfl_xor(mrow, 32));
      if (ok && g == 0) atomicMax(a.rowmax + r, __float_as_uint(mrow));
    }
  }
}

// ---------------------------------------------------------------------------
// Single-load form, for key ranges short enough that every score of the
// workgroup fits in registers (at most SL_WAVES x NT tiles). Eight wavefronts
// split the key tiles; each loads its tiles' K straight into registers in
// MFMA operand layout, forms and keeps the scores, then loads V into the same
// registers while the row maxima are exchanged through LDS. The probabilities
// are formed once, against the exact maximum, from the kept scores, so K and V
// cross the memory system once and the path has two memory round trips
// instead of one per tile.
//
// In the KV tile layout every K and V fragment a lane needs is its 16 bytes
// of one contiguous 1 KiB run: the loads are fully coalesced, and the scores
// of lane (c16, g) are keys 8 g .. 8 g + 7 of the tile, the keys of its V^T
// fragments.
constexpr int SL_WAVES = 8;

template <int D, int QB, int NT>
struct SlSmem {
  static constexpr int NDB = D / 16;
  static constexpr int OV = NDB * QB * 64;  // f32x4 partial-output values of one wavefront
};

template <int D, int QB, int NT>
__global__ __launch_bounds__(64 * SL_WAVES) void attn_sl_kernel(AttnArgs a) {
  constexpr int NDB = D / 16, NKK = D / 32;
  using SM = SlSmem<D, QB, NT>;
  __shared__ f32x4 s_o[SL_WAVES][SM::OV];
  __shared__ float s_max[SL_WAVES][QB * 16];
  __shared__ float s_l[SL_WAVES][QB * 16];
  const int h = blockIdx.x, br = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int kvh = h / (a.Hq / a.Hkv);
  const int L = a.L, P = a.P;
  const int pt = (P + KT - 1) / KT, bt = (L + KT - 1) / KT, T = pt + bt;
  const int t_lo = wv * T / SL_WAVES, nt = (wv + 1) * T / SL_WAVES - t_lo;  // nt <= NT
  const float sl2 = a.scale * 1.4426950408889634f;

  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;  // KV tile layout
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;

  // K of the wavefront's tiles (whole tiles; keys past a source's end are
  // masked below)
  u32x4 kv[NT][2][NKK];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    if (i >= nt) break;
    const int t = t_lo + i;
    const bool pre = t < pt;
    const uint16_t* kt = (pre ? kc : ks) + (int64_t)(pre ? t : t - pt) * KT * D + lane * 8;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) kv[i][kb][kk] = *(const u32x4*)(kt + (kb * NKK + kk) * 512);
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

  // scores S^T = K Q^T, kept: sc[i][qb][kb][j] is key p0 + 8 g + 4 kb + j of
  // tile i, query 16 qb + c16; masked keys -inf
  f32x4 sc[NT][QB][2];
  float mraw[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) mraw[qb] = -INFINITY;
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    if (i >= nt) break;
    const int t = t_lo + i;
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT, lim = pre ? P : L;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      int lq = lim;  // block-causal: rows 16 qb .. lie in one sub-block
      if (!pre && a.cblk) lq = min(lim, ((qb * 16) / a.cblk + 1) * a.cblk);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) acc = mfma16(kv[i][kb][kk], qf[qb][kk], acc);
        if (p0 + KT > lq) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[j] = p0 + 8 * g + 4 * kb + j < lq ? acc[j] : -INFINITY;
        }
        sc[i][qb][kb] = acc;
        mraw[qb] = max2(mraw[qb], max2(max2(acc[0], acc[1]), max2(acc[2], acc[3])));
      }
    }
  }
  // V^T of the same keys (the K registers are free now): lane (c16, g) takes
  // dims 16 db + c16, keys 8 g .. 8 g + 7
  u32x4 vf[NT][NDB];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    if (i >= nt) break;
    const int t = t_lo + i;
    const bool pre = t < pt;
    const uint16_t* vt = (pre ? vc : vs) + (int64_t)(pre ? t : t - pt) * KT * D + lane * 8;
#pragma unroll
    for (int db = 0; db < NDB; ++db) vf[i][db] = *(const u32x4*)(vt + db * 512);
  }

  // the exact row maximum over the eight wavefronts (the V loads stay in
  // flight across the barrier)
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float mw = pair32_max(pair16_max(mraw[qb]));
    if (g == 0) s_max[wv][qb * 16 + c16] = mw;
  }
  lds_barrier();
  float m[QB], l[QB];
  f32x4 o[NDB][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    float mx = s_max[0][qb * 16 + c16];
#pragma unroll
    for (int w = 1; w < SL_WAVES; ++w) mx = max2(mx, s_max[w][qb * 16 + c16]);
    m[qb] = mx * sl2;  // every probability 2^(s sl2 - m) <= 1
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // probabilities against the exact maximum; V meets them rounded to bf16
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    if (i >= nt) break;
    const int t = t_lo + i;
    const bool pre = t < pt;
    const int p0 = (pre ? t : t - pt) * KT, lim = pre ? P : L;
    if (p0 + KT > lim) {
      // zero V at keys past the end of the source (0 * inf would poison o)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int pos = p0 + 8 * g + 2 * e;
        const unsigned mk = (pos < lim ? 0xFFFFu : 0u) | (pos + 1 < lim ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int db = 0; db < NDB; ++db) vf[i][db][e] &= mk;
      }
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float nm = -m[qb];
      uint16_t pb[8];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = fast_exp2(__builtin_fmaf(sc[i][qb][kb][j], sl2, nm));  // -inf: 0
          l[qb] += p;
          pb[kb * 4 + j] = f2bf_bits(p);
        }
      const u32x4 pf = *(const u32x4*)pb;  // keys 8 g .. 8 g + 7
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db][qb] = mfma16(vf[i][db], pf, o[db][qb]);
    }
  }

  // the eight partial states share the maximum: they add up, in wavefront
  // order (deterministic); every thread then finishes a share of the outputs
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lw = pair32_sum(pair16_sum(l[qb]));
    if (g == 0) s_l[wv][qb * 16 + c16] = lw;
#pragma unroll
    for (int db = 0; db < NDB; ++db) s_o[wv][(db * QB + qb) * 64 + lane] = o[db][qb];
  }
  lds_barrier();
  // f = tid + 64 SL_WAVES i: every entry of a thread has the lane tid % 64 and
  // the row block (tid / 64) % QB, so a thread's entries are one row
  static_assert((64 * SL_WAVES) % (64 * QB) == 0, "a thread's entries share their row");
  float mrow = 0.f;  // largest |stored value| of this thread's part of its row
  for (int f = tid; f < SM::OV; f += 64 * SL_WAVES) {
    const int ln = f & 63, qb = (f >> 6) % QB, db = (f >> 6) / QB;
    const int q16 = ln & 15, g4 = ln >> 4;
    const int row = qb * 16 + q16;
    if (row >= L) continue;
    f32x4 acc = s_o[0][f];
    float ls = s_l[0][qb * 16 + q16];
#pragma unroll
    for (int w = 1; w < SL_WAVES; ++w) {
      acc += s_o[w][f];
      ls += s_l[w][qb * 16 + q16];
    }
    const float inv = 1.0f / ls;
    uint16_t ob[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ob[j] = f2bf_bits(acc[j] * inv);
      mrow = fmaxf(mrow, fabsf(bf2f_bits(ob[j])));
    }
    const int col = h * D + db * 16 + g4 * 4;
    *(uint2*)(a.out + packA_off(br * L + row, col, a.Mp)) = *(const uint2*)ob;
  }
  if (a.rowmax) {
    // over the row's 4 column groups (lanes q16 + 16 g4), then over the
    // wavefronts of the same row block (through LDS, reusing s_l: every
    // thread has read it above), one atomic per row
    mrow = fmaxf(mrow, __shfl_xor(mrow, 16));
    mrow = fmaxf(mrow, __shfl_xor(mrow, 32));
    lds_barrier();
    float* s_m = &s_l[0][0];
    if (lane < 16) s_m[wv * 16 + lane] = mrow;
    lds_barrier();
    if (tid < 16 * QB) {
      const int qb = tid >> 4, row = qb * 16 + (tid & 15);
      float m = 0.f;
      for (int w = qb; w < SL_WAVES; w += QB) m = fmaxf(m, s_m[w * 16 + (tid & 15)]);
      if (row < L) atomicMax(a.rowmax + br * L + row, __float_as_uint(m));
    }
  }
}

template <int D, int QB>
hipError_t launch_sl(const AttnArgs& a, int nt, hipStream_t s) {
  const dim3 grid(a.Hq, a.nb), block(64 * SL_WAVES);
  switch (nt) {
    case 1: hipLaunchKernelGGL((attn_sl_kernel<D, QB, 1>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_sl_kernel<D, QB, 2>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((attn_sl_kernel<D, QB, 3>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Grouped form, for key ranges too long for the single-load form (more than
// SL_WAVES x 3 tiles) with grouped-query heads (2..8 query heads per KV head).
// The keys are cut into NS splits; a workgroup takes one (KV head, branch,
// split) with one wavefront per query head of the group, so that every K / V
// tile crosses into the CU once for all the group's heads (wavefront 0 copies
// it into an LDS ring, the others read it after a barrier). Three launches:
//   gmax   each row's largest score over the split's keys,
//   gpv    the exact row maximum (over the splits), then the probabilities
//          rounded to bf16 against it, their sum and P V over the split,
//   merge  the splits' sums and outputs added in split order, normalised,
//          rounded to bf16 into the packed operand of the output projection.
// The scores are formed the same way (the same MFMA chain, tile by tile) in
// gmax and gpv, so the maximum gpv subtracts is exactly one of its scores.
constexpr int GQ_RING = 4;  // LDS slots: one tile in use, GQ_RING - 1 in flight

struct GroupSplit {
  int p_lo, np, n;  // first prefix tile; prefix tiles; all tiles (the last split
                    // also takes the block's tiles)
};
__device__ __forceinline__ GroupSplit group_split(int P, int L, int sp, int NS) {
  const int pt = (P + KT - 1) / KT, bt = (L + KT - 1) / KT;
  const int p_lo = sp * pt / NS, p_hi = (sp + 1) * pt / NS;
  return {p_lo, p_hi - p_lo, p_hi - p_lo + (sp == NS - 1 ? bt : 0)};
}

template <int D, int QB, bool WITH_V>
__device__ __forceinline__ void group_issue(const AttnArgs& a, const GroupSplit& gs, int i,
                                            int slot, uint32_t ring, const uint16_t* kc,
                                            const uint16_t* vc, const uint16_t* ks,
                                            const uint16_t* vs, int lane) {
  using T = TileLds<D>;
  constexpr int OPS = WITH_V ? T::OPS : 2 * (D / 32);
  constexpr int SLOT = WITH_V ? T::TILE : T::KBYTES;
  i = i < gs.n ? i : gs.n - 1;  // past the last tile: the last one again
  const bool pre = i < gs.np;
  const int64_t off = (int64_t)(pre ? gs.p_lo + i : i - gs.np) * KT * D;
  const uint32_t sb = ring + (uint32_t)slot * SLOT;
#pragma unroll
  for (int q = 0; q < OPS; ++q) tile_copy<D>(q, (pre ? kc : ks) + off, (pre ? vc : vs) + off, sb, lane);
}

// Q^T operand of query head h, rows 16 qb + c16 of branch br (zero past L)
template <int D, int QB>
__device__ __forceinline__ void group_q(const AttnArgs& a, int br, int h, int c16, int g,
                                        u32x4 (&qf)[QB][D / 32]) {
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qb * 16 + c16;
    const uint16_t* qrow = a.q + (((int64_t)br * a.Hq + h) * a.L + (row < a.L ? row : 0)) * D;
    const unsigned keep = row < a.L ? ~0u : 0u;
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
      qf[qb][kk] = *(const u32x4*)(qrow + kk * 32 + g * 8) & keep;
  }
}

// scratch layout: mpart [nb][Hq][L][NS], lsum [NS][nb][Hq][L], opart [NS][nb][Hq][L][D]
struct GroupScratch {
  float *m, *l, *o;
};
__host__ __device__ __forceinline__ size_t group_scratch_floats(const AttnArgs& a, int NS) {
  const size_t rows = (size_t)a.nb * a.Hq * a.L;
  return rows * NS * 2 + rows * NS * a.d;
}
__device__ __forceinline__ GroupScratch group_scratch(const AttnArgs& a, int NS) {
  const size_t rows = (size_t)a.nb * a.Hq * a.L;
  return {a.scratch, a.scratch + rows * NS, a.scratch + rows * NS * 2};
}

template <int D, int QB>
__global__ __launch_bounds__(512) void attn_gmax_kernel(AttnArgs a, int NS) {
  using T = TileLds<D>;
  constexpr int KOPS = 2 * (D / 32);
  __shared__ __attribute__((aligned(1024))) char smem[GQ_RING * T::KBYTES];
  const int kvh = blockIdx.x, br = blockIdx.y, sp = blockIdx.z;
  const int G = a.Hq / a.Hkv;
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = kvh * G + wv, g = lane >> 4, c16 = lane & 15;
  const GroupSplit gs = group_split(a.P, a.L, sp, NS);
  const int np = gs.np;
  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;
  const uint32_t ring = (uint32_t)(uintptr_t)smem;
  if (wv == 0 && gs.n > 0)
#pragma unroll
    for (int i = 0; i < GQ_RING - 1; ++i)
      group_issue<D, QB, false>(a, gs, i, i, ring, kc, vc, ks, vs, lane);
  u32x4 qf[QB][D / 32];
  group_q<D, QB>(a, br, h, c16, g, qf);
  float mraw[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) mraw[qb] = -INFINITY;
  for (int i = 0; i < gs.n; ++i) {
    if (wv == 0) attn_wait_vmcnt<KOPS * (GQ_RING - 2)>();  // tile i has landed
    lds_barrier();  // ... for every wavefront, which all finished tile i - 1
    if (wv == 0)
      group_issue<D, QB, false>(a, gs, i + GQ_RING - 1, (i + GQ_RING - 1) % GQ_RING, ring, kc, vc,
                                ks, vs, lane);
    const bool pre = i < np;
    tile_max<D, QB>(smem + (i % GQ_RING) * T::KBYTES, lane, qf, mraw,
                    (pre ? gs.p_lo + i : i - np) * KT, pre ? a.P : a.L, g, pre ? 0 : a.cblk, 0);
  }
  if (wv == 0) attn_wait_vmcnt<0>();
  const GroupScratch sc = group_scratch(a, NS);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float m = pair32_max(pair16_max(mraw[qb]));
    const int row = qb * 16 + c16;
    if (g == 0 && row < a.L) sc.m[(((int64_t)br * a.Hq + h) * a.L + row) * NS + sp] = m;
  }
}

template <int D, int QB>
__global__ __launch_bounds__(512) void attn_gpv_kernel(AttnArgs a, int NS) {
  using T = TileLds<D>;
  constexpr int NDB = D / 16;
  __shared__ __attribute__((aligned(1024))) char smem[GQ_RING * T::TILE];
  const int kvh = blockIdx.x, br = blockIdx.y, sp = blockIdx.z;
  const int G = a.Hq / a.Hkv;
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = kvh * G + wv, g = lane >> 4, c16 = lane & 15;
  const GroupSplit gs = group_split(a.P, a.L, sp, NS);
  const int np = gs.np;
  const float sl2 = a.scale * 1.4426950408889634f;
  const uint16_t* kc = a.kcache + (int64_t)kvh * D * a.vld;
  const uint16_t* vc = a.vcache + (int64_t)kvh * D * a.vld;
  const int64_t st_base = (((int64_t)br * a.layers + a.layer) * 2) * a.Hkv;
  const uint16_t* ks = a.staging + (st_base + 0 * a.Hkv + kvh) * D * a.vlds;
  const uint16_t* vs = a.staging + (st_base + 1 * a.Hkv + kvh) * D * a.vlds;
  const uint32_t ring = (uint32_t)(uintptr_t)smem;
  if (wv == 0 && gs.n > 0)
#pragma unroll
    for (int i = 0; i < GQ_RING - 1; ++i)
      group_issue<D, QB, true>(a, gs, i, i, ring, kc, vc, ks, vs, lane);
  u32x4 qf[QB][D / 32];
  group_q<D, QB>(a, br, h, c16, g, qf);
  const GroupScratch sc = group_scratch(a, NS);
  float m[QB], l[QB];
  f32x4 o[NDB][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = qb * 16 + c16;
    float mx = 0.f;  // rows past L: zero queries, any finite reference
    if (row < a.L) {
      const float* mp = sc.m + (((int64_t)br * a.Hq + h) * a.L + row) * NS;
      mx = mp[0];
      for (int s2 = 1; s2 < NS; ++s2) mx = max2(mx, mp[s2]);
    }
    m[qb] = mx * sl2;  // the exact row maximum: every probability <= 1
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int i = 0; i < gs.n; ++i) {
    if (wv == 0) attn_wait_vmcnt<T::OPS * (GQ_RING - 2)>();
    lds_barrier();
    if (wv == 0)
      group_issue<D, QB, true>(a, gs, i + GQ_RING - 1, (i + GQ_RING - 1) % GQ_RING, ring, kc, vc,
                               ks, vs, lane);
    AttnTile<D> x;
    tile_fetch<D>(smem + (i % GQ_RING) * T::TILE, lane, x);
    const bool pre = i < np;
    tile_update<D, QB, false>(x, qf, m, l, o, (pre ? gs.p_lo + i : i - np) * KT,
                              pre ? a.P : a.L, sl2, g, pre ? 0 : a.cblk, 0);
  }
  if (wv == 0) attn_wait_vmcnt<0>();
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float ls = pair32_sum(pair16_sum(l[qb]));
    const int row = qb * 16 + c16;
    if (row >= a.L) continue;
    const int64_t r = (((int64_t)sp * a.nb + br) * a.Hq + h) * a.L + row;
    if (g == 0) sc.l[r] = ls;
#pragma unroll
    for (int db = 0; db < NDB; ++db) *(f32x4*)(sc.o + r * D + db * 16 + g * 4) = o[db][qb];
  }
}

// one thread per (branch, head, row, 4 dimensions)
template <int D>
__global__ __launch_bounds__(256) void attn_gmerge_kernel(AttnArgs a, int NS) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int q4 = (int)(t % (D / 4));
  const int64_t rr = t / (D / 4);  // (branch, head, row)
  const bool ok = rr < (int64_t)a.nb * a.Hq * a.L;
  const int64_t r = ok ? rr : 0;
  const int row = (int)(r % a.L), h = (int)((r / a.L) % a.Hq), br = (int)(r / ((int64_t)a.L * a.Hq));
  const GroupScratch sc = group_scratch(a, NS);
  const int64_t rows = (int64_t)a.nb * a.Hq * a.L;
  f32x4 acc = *(const f32x4*)(sc.o + r * D + q4 * 4);
  float ls = sc.l[r];
  for (int s2 = 1; s2 < NS; ++s2) {
    acc += *(const f32x4*)(sc.o + (s2 * rows + r) * D + q4 * 4);
    ls += sc.l[s2 * rows + r];
  }
  const float inv = 1.0f / ls;
  uint16_t ob[4];
  float mrow = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    ob[j] = f2bf_bits(acc[j] * inv);
    mrow = fmaxf(mrow, fabsf(bf2f_bits(ob[j])));
  }
  if (ok) *(uint2*)(a.out + packA_off(br * a.L + row, h * D + q4 * 4, a.Mp)) = *(const uint2*)ob;
  if (a.rowmax) {  // the D / 4 threads of one (branch, head, row) are adjacent lanes
#pragma unroll
    for (int o = 1; o < D / 4; o <<= 1) mrow = fmaxf(mrow, __shfl_xor(mrow, o));
    if (ok && q4 == 0) atomicMax(a.rowmax + br * a.L + row, __float_as_uint(mrow));
  }
}

// key splits of the grouped form before the per-call caps: enough workgroups
// for the chip's 256 CUs, at most 16
int group_splits(int nb, int Hkv) {
  return std::min(16, std::max(1, (256 + Hkv * nb - 1) / (Hkv * nb)));
}

template <int D>
hipError_t launch_group(const AttnArgs& a, int NS, hipStream_t s) {
  const int G = a.Hq / a.Hkv;
  const dim3 grid(a.Hkv, a.nb, NS), block(64 * G);
  if (a.L <= 16) {
    hipLaunchKernelGGL((attn_gmax_kernel<D, 1>), grid, block, 0, s, a, NS);
    hipLaunchKernelGGL((attn_gpv_kernel<D, 1>), grid, block, 0, s, a, NS);
  } else {
    hipLaunchKernelGGL((attn_gmax_kernel<D, 2>), grid, block, 0, s, a, NS);
    hipLaunchKernelGGL((attn_gpv_kernel<D, 2>), grid, block, 0, s, a, NS);
  }
  const int64_t threads = (int64_t)a.nb * a.Hq * a.L * (D / 4);
  hipLaunchKernelGGL((attn_gmerge_kernel<D>), dim3((unsigned)((threads + 255) / 256)), dim3(256),
                     0, s, a, NS);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnArgs& a, hipStream_t s) {
  const int T = (a.P + KT - 1) / KT + (a.L + KT - 1) / KT;
  const int nt = (T + SL_WAVES - 1) / SL_WAVES;  // most tiles of one wavefront
  if (a.L <= 32 && nt <= 3) {
    if (a.L <= 16) return launch_sl<D, 1>(a, nt, s);
    return launch_sl<D, 2>(a, nt, s);
  }
  const int G = a.Hq / a.Hkv;
  if (a.L <= 32 && G >= 2 && G <= 8 && a.scratch) {
    // key splits: enough workgroups for the chip, at least 4 prefix tiles each,
    // within the scratch
    const int pt = (a.P + KT - 1) / KT;
    int NS = group_splits(a.nb, a.Hkv);
    NS = std::min(NS, std::max(1, pt / 4));
    while (NS > 1 && group_scratch_floats(a, NS) * 4 > a.scratch_bytes) --NS;
    if (group_scratch_floats(a, NS) * 4 <= a.scratch_bytes) return launch_group<D>(a, NS, s);
  }
  // up to 64 query rows per workgroup; longer blocks (multi-block windows) in
  // groups of 64 rows, each group reading all of the branch's keys
  const dim3 grid(a.Hq, a.nb, (a.L + 63) / 64);
  switch (a.L > 64 ? 4 : (a.L + 15) / 16) {
    case 1: hipLaunchKernelGGL((attn_kernel<D, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_kernel<D, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((attn_kernel<D, 3>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((attn_kernel<D, 4>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

size_t attention_scratch_bytes(int nb, int L, int Hq, int Hkv, int d) {
  const int G = Hkv > 0 ? Hq / Hkv : 0;
  if (L > 32 || G < 2 || G > 8) return 0;
  const size_t rows = (size_t)nb * Hq * L;
  return rows * group_splits(nb, Hkv) * (2 + (size_t)d) * 4;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.L < 1 || a.L > 256 || a.P < 0 || a.Hq % a.Hkv || a.vld % KT || a.vlds % KT ||
      a.L > a.vlds || a.P > a.vld)
    return hipErrorInvalidValue;
  if (a.cblk < 0 || (a.cblk > 0 && (a.cblk % 16 || a.L % a.cblk))) return hipErrorInvalidValue;
  if (a.d == 128) return launch_d<128>(a, s);
  if (a.d == 64) return launch_d<64>(a, s);
  return hipErrorInvalidValue;
}

// Weight-streaming bf16 GEMM for the skinny row counts of the verify step
// (M = branches x block rows) with fused epilogues:
//   EPI_QKV    bias + rotate-half RoPE on q/k, q -> attention input, k/v -> the
//              branch K/V staging (the Pre-Write of Sec. 3.4)
//   EPI_RESID  residual add into the fp32 residual stream (O-proj, down-proj)
//   EPI_SWIGLU silu(gate) * up -> packed bf16 operand of the down projection
//   EPI_LMHEAD per (row, 128-token tile) softmax partials: max, argmax, sum exp
//              (the logits never reach memory)
//
// Work decomposition. A workgroup (4 wavefronts) covers one 256-row tile of the
// activations (each wavefront 64 rows x 128 output columns), so every weight
// byte is read from HBM once per row tile. The (column tile, 64-wide k-chunk)
// iteration space is split evenly over the column workgroups (stream-K): every
// CU streams the same number of weight bytes whatever the tile count. A tile
// covered by one workgroup runs its epilogue in place; a tile split over
// several writes per-workgroup partial sums, which gemm_fixup_kernel adds in
// workgroup order (deterministic) after the kernel boundary and then runs the
// epilogue. No workgroup waits for another. The QKV epilogue (bias, RoPE,
// scatter to q / K / V staging) always runs in the fix-up kernel, which keeps
// its register-heavy code out of the streaming loop.
//
// Pipeline. Per iteration (a 64-wide k-chunk) the 16 KiB weight chunk goes
// straight from global memory into a 4-slot LDS ring (LDS-DMA, no registers)
// and each wavefront's 8 activation fragments (L2-resident) into one of three
// register sets, both three iterations ahead (the in-order vmcnt queue makes
// equal lead distances the only way not to wait on younger loads).
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

template <int D>
__device__ __forceinline__ void qkv_epilogue(const GemmArgs& a, f32x4 (&acc)[4][8], int tile,
                                             int row0, int lane, unsigned nbmask) {
  constexpr int HD = D / 2, HALF_NB = HD / 16;  // RoPE partner offset in 16-column blocks
  const int g = lane >> 4, c16 = lane & 15;
  const int qcols = a.Hq * D, kcols = a.Hkv * D;
  // A 128-column tile never straddles the q / k / v sections (their widths are
  // multiples of 128) and holds whole heads, so the section is per tile.
  const int n0 = tile * LOPA_BN;
  const int sect = n0 < qcols ? 0 : (n0 < qcols + kcols ? 1 : 2);
  const int base = sect == 0 ? 0 : (sect == 1 ? qcols : qcols + kcols);
  if (n0 >= a.N) return;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = row0 + mb * 16 + g * 4 + j;
      if (r >= a.M) continue;
      const int br = r / a.L, i = r % a.L;
      const float* cs_row = a.rope + (int64_t)(a.P + i) * HD * 2;
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        if (!((nbmask >> nb) & 1)) continue;
        const bool low = (nb % (D / 16)) < HALF_NB;
        if (sect < 2 && !low) continue;  // written together with its partner
        const int nl = n0 - base + nb * 16 + c16;
        const int head = nl / D, dim = nl % D;
        const int n = n0 + nb * 16 + c16;
        float o1 = acc[mb][nb][j] + (a.bias ? a.bias[n] : 0.f), o2 = 0.f;
        if (sect < 2) {
          const float x2 = acc[mb][(nb + HALF_NB) & 7][j] + (a.bias ? a.bias[n + HD] : 0.f);
          const float2 cs = *(const float2*)(cs_row + dim * 2);
          const float x1 = o1;
          o1 = x1 * cs.x - x2 * cs.y;
          o2 = x2 * cs.x + x1 * cs.y;
        }
        if (sect == 0) {
          uint16_t* q = a.q_out + (((int64_t)br * a.Hq + head) * a.L + i) * D;
          q[dim] = f2bf_bits(o1);
          q[dim + HD] = f2bf_bits(o2);
        } else {
          uint16_t* st = a.staging +
                         (((((int64_t)br * a.layers + a.layer) * 2 + (sect - 1)) * a.Hkv + head) *
                              a.Lcap + i) * D;
          st[dim] = f2bf_bits(o1);
          if (sect == 1) st[dim + HD] = f2bf_bits(o2);
        }
      }
    }
}

template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, f32x4 (&acc)[4][8], int tile, int row0,
                                         int lane, uint16_t* stage, unsigned nbmask = 0xffu) {
  const int g = lane >> 4, c16 = lane & 15;
  if constexpr (EPI == EPI_RESID) {
    #pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      #pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = row0 + mb * 16 + g * 4 + j;
        if (r >= a.M) continue;
        float* xr = a.x + (int64_t)r * a.N + tile * LOPA_BN + c16;
        #pragma unroll
        for (int nb = 0; nb < 8; ++nb)
          if ((nbmask >> nb) & 1) xr[nb * 16] += acc[mb][nb][j];
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // gate in columns 0..63, up in 64..127 of the tile; output columns
    // [64 tile, 64 tile + 64). Stage through LDS so each lane writes 16 bytes.
    uint16_t* e = stage;  // this wavefront's 64 x 72 staging tile
    #pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      #pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        #pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (!((nbmask >> nb) & 1)) continue;
          const float gt = acc[mb][nb][j], up = acc[mb][nb + 4][j];
          const float h = gt / (1.0f + expf(-gt)) * up;
          e[(mb * 16 + g * 4 + j) * 72 + nb * 16 + c16] = f2bf_bits(h);
        }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): wave-local LDS writes done
    __builtin_amdgcn_wave_barrier();
    const int Nout = a.N >> 1;
    #pragma unroll
    for (int q = lane; q < 64 * 8; q += 64) {
      const int rr = q >> 3, cg = q & 7;
      const int r = row0 + rr;
      if (r >= a.M || !((nbmask >> (cg >> 1)) & 1)) continue;
      const uint4 v = *(const uint4*)(e + rr * 72 + cg * 8);
      *(uint4*)(a.a_out + packA_off(r, tile * 64 + cg * 8, a.Mp)) = v;
    }
    (void)Nout;
  } else if constexpr (EPI == EPI_LMHEAD) {
    #pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      #pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = row0 + mb * 16 + g * 4 + j;
        float m = -INFINITY;
        int mi = 0x7fffffff;
        float v[8];
        #pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
          const int col = tile * LOPA_BN + nb * 16 + c16;
          v[nb] = (col < a.vocab && col != a.mask_id) ? acc[mb][nb][j] : -INFINITY;
          if (v[nb] > m) { m = v[nb]; mi = col; }
        }
        #pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float om = __shfl_xor(m, o);
          const int oi = __shfl_xor(mi, o);
          if (om > m || (om == m && oi < mi)) { m = om; mi = oi; }
        }
        float s = 0.f;
        if (m != -INFINITY)
          #pragma unroll
          for (int nb = 0; nb < 8; ++nb) s += expf(v[nb] - m);
        #pragma unroll
        for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o);
        if (c16 == 0 && r < a.M) {
          const int64_t o = (int64_t)r * a.tiles + tile;
          a.pm[o] = m;
          a.ps[o] = s;
          a.pi[o] = mi;
        }
      }
  } else {  // EPI_QKV
    if (a.d == 128) qkv_epilogue<128>(a, acc, tile, row0, lane, nbmask);
    else qkv_epilogue<64>(a, acc, tile, row0, lane, nbmask);
  }
}

__device__ __forceinline__ int64_t sk_start(int g, int64_t I, int G) { return (int64_t)g * I / G; }

// workgroup whose range contains iteration j
__device__ __forceinline__ int sk_owner(int64_t j, int64_t I, int G) {
  int g = (int)((j * G) / I);
  while (g + 1 < G && sk_start(g + 1, I, G) <= j) ++g;
  while (g > 0 && sk_start(g, I, G) > j) --g;
  return g;
}

// partial-sum slot of contributor gc of a tile that starts at iteration t0
__device__ __forceinline__ int sk_slot(int gc, int g_lo, int64_t t0, int64_t I, int G) {
  return (gc == g_lo && sk_start(gc, I, G) < t0) ? 2 * gc + 1 : 2 * gc;
}

constexpr int GEMM_THREADS = 256;
constexpr int W_SLOTS = 4;  // LDS ring of 16 KiB weight chunks (three in flight)

// Asynchronous global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane l writes bytes [16 l, 16 l + 16) of the 1 KiB LDS block at lds_addr
// (wave-uniform, passed in M0). The compiler does not track it: completion is
// awaited with an explicit vmcnt wait before the workgroup barrier.
__device__ __forceinline__ void lds_dma16(const void* gptr, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_addr), "v"(gptr)
               : "memory");
}

// weight chunk of iteration itx -> ring slot (4 x 1 KiB blocks per wavefront)
#define GEMM_DMA_W(itx)                                                                  \
  {                                                                                      \
    const uint32_t slot_ = sW_base + (uint32_t)(((itx) % W_SLOTS) * 16384);              \
    const char* src_ = (const char*)a.W + (int64_t)(itx) * 16384 + lane * 16;            \
    _Pragma("unroll") for (int r_ = 0; r_ < 4; ++r_) {                                   \
      const int blk_ = r_ * 4 + wv;                                                      \
      lds_dma16(src_ + blk_ * 1024, slot_ + blk_ * 1024);                                \
    }                                                                                    \
  }
// this wavefront's 8 activation fragments of 64-wide chunk kcx -> registers
#define GEMM_LOAD_A(dst, kcx)                                                            \
  _Pragma("unroll") for (int kk_ = 0; kk_ < 2; ++kk_)                                    \
    _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                                  \
      dst[kk_ * 4 + mb_] = A[((int64_t)((2 * (kcx) + kk_) * RB + rb0 + mb_)) * 64 + lane];
#define GEMM_ZERO_ACC()                                                                  \
  _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                                    \
    _Pragma("unroll") for (int nb_ = 0; nb_ < 8; ++nb_) acc[mb_][nb_] = f32x4{0.f, 0.f, 0.f, 0.f};

// One iteration it. Every iteration j issues, in this order, the 8 activation
// loads then the 4 weight copies of iteration j + 3 (the prologue issues those
// of it0 .. it0 + 2 the same way). When iteration it starts, what was issued
// after the weight copies of `it` is iterations it + 1 and it + 2: 24
// operations (fewer near the end of the range), so vmcnt(24) means both the
// weights and the activations of `it` have arrived.
#define GEMM_STEP(ar)                                                                    \
  {                                                                                      \
    if (it + 2 < it1) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");                  \
    else if (it + 1 < it1) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");             \
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");                                \
    lds_barrier();                                                                       \
    const u32x4* wl_ = sW + (int)(it % W_SLOTS) * 1024;                                  \
    _Pragma("unroll") for (int kk_ = 0; kk_ < 2; ++kk_)                                  \
      _Pragma("unroll") for (int nb_ = 0; nb_ < 8; ++nb_) {                              \
        const u32x4 bf_ = wl_[(kk_ * 8 + nb_) * 64 + lane];                              \
        _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                              \
          acc[mb_][nb_] = mfma16(ar[kk_ * 4 + mb_], bf_, acc[mb_][nb_]);                 \
      }                                                                                  \
    if (it + 3 < it1) {                                                                  \
      GEMM_LOAD_A(ar, (int)((it + 3) % KC));                                             \
      GEMM_DMA_W(it + 3);                                                                \
    }                                                                                    \
  }

#define GEMM_ROTATE()                                                                    \
  _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                     \
    const u32x4 t_ = a0[i_];                                                             \
    a0[i_] = a1[i_];                                                                     \
    a1[i_] = a2[i_];                                                                     \
    a2[i_] = t_;                                                                         \
  }

template <int EPI>
__global__ __launch_bounds__(GEMM_THREADS, 1) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) u32x4 sW[W_SLOTS * 1024];  // ring of 16 KiB chunks
  __shared__ __attribute__((aligned(16))) uint16_t sE[4][EPI == EPI_SWIGLU ? 64 * 72 : 8];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t sW_base = (uint32_t)(uintptr_t)sW;
  const int MT = a.mtiles;
  const int G = a.grid / MT;
  // Hardware places workgroup b on XCD b % 8; each XCD gets a contiguous piece
  // of the logical index q, so neighbouring iteration ranges share an L2 and
  // the row tiles of one column workgroup stream the same weights together.
  const int b = blockIdx.x;
  const int q = (a.grid % 8 == 0) ? (b & 7) * (a.grid >> 3) + (b >> 3) : b;
  const int mt = q % MT, g = q / MT;
  const int KC = a.KC;
  const int64_t I = (int64_t)a.tiles * KC;
  const int64_t it0 = sk_start(g, I, G), it1 = sk_start(g + 1, I, G);
  if (it0 >= it1) return;
  const int RB = a.Mp >> 4;
  const int rb0 = mt * 16 + wv * 4;     // first 16-row block of this wavefront
  const int row0 = mt * 256 + wv * 64;  // first row of this wavefront
  const u32x4* __restrict__ A = (const u32x4*)a.A;

  f32x4 acc[4][8];
  // activation register sets: iteration j uses set (j - it0) % 3 (after the
  // rotations below, the set named a0 serves the current iteration)
  u32x4 a0[8], a1[8], a2[8];
  GEMM_LOAD_A(a0, (int)(it0 % KC));
  GEMM_DMA_W(it0);
  if (it0 + 1 < it1) {
    GEMM_LOAD_A(a1, (int)((it0 + 1) % KC));
    GEMM_DMA_W(it0 + 1);
  }
  if (it0 + 2 < it1) {
    GEMM_LOAD_A(a2, (int)((it0 + 2) % KC));
    GEMM_DMA_W(it0 + 2);
  }
  // Segments: the iterations of one column tile inside [it0, it1).
  int64_t it = it0;
  while (it < it1) {
    const int64_t seg0 = it;
    const int tile = (int)(it / KC);
    const int64_t seg1 = (it1 < (int64_t)(tile + 1) * KC) ? it1 : (int64_t)(tile + 1) * KC;
    GEMM_ZERO_ACC();
    for (;;) {
      GEMM_STEP(a0);
      if (++it >= seg1) { GEMM_ROTATE(); break; }
      GEMM_STEP(a1);
      if (++it >= seg1) { GEMM_ROTATE(); GEMM_ROTATE(); break; }
      GEMM_STEP(a2);
      if (++it >= seg1) break;
    }
    if (EPI != EPI_QKV && seg0 % KC == 0 && seg1 % KC == 0) {
      epilogue<EPI>(a, acc, tile, row0, lane, sE[wv]);
    } else {
      const int slot = (2 * g + (seg0 == it0 ? 0 : 1)) * MT + mt;
      f32x4* part = (f32x4*)a.partials + ((int64_t)slot * 4 + wv) * 32 * 64;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) part[(mb * 8 + nb) * 64 + lane] = acc[mb][nb];
    }
  }
  // nothing may still be writing LDS when the workgroup ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Sum the partial tiles of split tiles in workgroup order and run the epilogue.
// One wavefront per (column tile, row tile, 64-row block, column group): the
// groups pair the 16-column blocks an epilogue couples (RoPE halves, gate/up),
// nb and nb + PAIR; the LM-head epilogue reduces over all 8 blocks of a row,
// so it takes one group. Whole tiles (done in gemm_kernel) return at once.
template <int EPI>
__global__ __launch_bounds__(64) void gemm_fixup_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sE[EPI == EPI_SWIGLU ? 64 * 72 : 8];
  constexpr int GROUPS = EPI == EPI_LMHEAD ? 1 : 4;
  const int MT = a.mtiles;
  const int G = a.grid / MT;
  int bid = blockIdx.x;
  const int cg = bid % GROUPS;
  bid /= GROUPS;
  const int w = bid % 4;
  bid /= 4;
  const int mt = bid % MT, tile = bid / MT;
  const int KC = a.KC;
  const int64_t I = (int64_t)a.tiles * KC;
  const int64_t t0 = (int64_t)tile * KC;
  const int g_lo = sk_owner(t0, I, G), g_hi = sk_owner(t0 + KC - 1, I, G);
  if (g_lo == g_hi && EPI != EPI_QKV) return;
  const int lane = threadIdx.x;
  const int row0 = mt * 256 + w * 64;
  const int pair = (EPI == EPI_QKV && a.d == 64) ? 2 : 4;
  const int nb_a = (cg % pair) + (cg / pair) * 2 * pair;
  const unsigned mask = GROUPS == 1 ? 0xffu : ((1u << nb_a) | (1u << (nb_a + pair)));
  f32x4 acc[4][8];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int gc = g_lo; gc <= g_hi; ++gc) {
    const int slot = sk_slot(gc, g_lo, t0, I, G) * MT + mt;
    const f32x4* p = (const f32x4*)a.partials + ((int64_t)slot * 4 + w) * 32 * 64;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
        if ((mask >> nb) & 1) acc[mb][nb] += p[(mb * 8 + nb) * 64 + lane];
  }
  epilogue<EPI>(a, acc, tile, row0, lane, sE, mask);
}

template <int EPI>
hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(gemm_kernel<EPI>, dim3(a.grid), dim3(GEMM_THREADS), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // split tiles exist unless every column workgroup owns whole tiles
  const int G = a.grid / a.mtiles;
  if (EPI == EPI_QKV || (int64_t)a.tiles * a.KC % G != 0 ||
      ((int64_t)a.tiles * a.KC / G) % a.KC != 0) {
    const int groups = EPI == EPI_LMHEAD ? 1 : 4;
    hipLaunchKernelGGL(gemm_fixup_kernel<EPI>, dim3(a.tiles * a.mtiles * 4 * groups), dim3(64), 0,
                       s, a);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, s);
    case EPI_LMHEAD: return launch_epi<EPI_LMHEAD>(a, s);
  }
  return hipErrorInvalidValue;
}

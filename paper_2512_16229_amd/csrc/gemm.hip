// Weight-streaming bf16 GEMM for the skinny row counts of the verify step
// (M = branches x block = 32 .. 512 rows) with fused epilogues:
//   EPI_QKV    bias + rotate-half RoPE on q/k, q -> attention input, k/v -> the
//              branch K/V staging (the Pre-Write of Sec. 3.4)
//   EPI_RESID  residual add into the fp32 residual stream (O-proj, down-proj)
//   EPI_SWIGLU silu(gate) * up -> packed bf16 operand of the down projection
//   EPI_LMHEAD per (row, 128-token tile) softmax partials: max, argmax, sum exp
//              (the logits never reach memory)
//
// Work decomposition: one workgroup covers all Mp rows (Mp/64 wavefronts, each
// 64 rows x 128 columns of a tile) so every weight byte is read from HBM once.
// The (tile, k-chunk) iteration space is split evenly over `grid` workgroups
// (stream-K), so all CUs stream weights even when N has few tiles. A tile split
// over several workgroups is finished by the last one to arrive (atomic
// counter): it sums the partial tiles in workgroup order, so the result does
// not depend on arrival order, and then runs the epilogue.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

__device__ __forceinline__ int64_t sk_start(int g, int64_t I, int G) { return (int64_t)g * I / G; }

// workgroup whose range contains iteration j
__device__ __forceinline__ int sk_owner(int64_t j, int64_t I, int G) {
  int g = (int)((j * G) / I);
  while (g + 1 < G && sk_start(g + 1, I, G) <= j) ++g;
  while (g > 0 && sk_start(g, I, G) > j) --g;
  return g;
}

template <int WAVES>
struct Smem {
  u32x4 w[2][1024];                 // two 16 KiB weight chunks
  uint16_t e[WAVES][64 * 72];       // per-wave epilogue staging (64 rows x 64 cols + pad)
  int flag;
};

template <int D>
__device__ __forceinline__ void qkv_epilogue(const GemmArgs& a, f32x4 (&acc)[4][8], int tile,
                                             int row0, int lane) {
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

template <int EPI, int WAVES>
__device__ __forceinline__ void epilogue(const GemmArgs& a, f32x4 (&acc)[4][8], int tile, int row0,
                                         int wv, int lane, Smem<WAVES>& sm) {
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
        for (int nb = 0; nb < 8; ++nb) xr[nb * 16] += acc[mb][nb][j];
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // gate in columns 0..63, up in 64..127 of the tile; output columns
    // [64 tile, 64 tile + 64). Stage through LDS so each lane writes 16 bytes.
    uint16_t* e = sm.e[wv];
    #pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      #pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        #pragma unroll
        for (int j = 0; j < 4; ++j) {
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
      if (r >= a.M) continue;
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
    if (a.d == 128) qkv_epilogue<128>(a, acc, tile, row0, lane);
    else qkv_epilogue<64>(a, acc, tile, row0, lane);
  }
}

// weights of iteration itx -> registers (this thread's share of the 16 KiB chunk)
#define GEMM_LOAD_W(dst, itx)                                                \
  _Pragma("unroll") for (int r_ = 0; r_ < NL; ++r_)                          \
    dst[r_] = W[(int64_t)(itx) * 1024 + r_ * NT + tid];
// this wavefront's 8 activation fragments of k-chunk kcx -> registers
#define GEMM_LOAD_A(dst, kcx)                                                \
  _Pragma("unroll") for (int kk_ = 0; kk_ < 2; ++kk_)                        \
    _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                      \
      dst[kk_ * 4 + mb_] = A[((int64_t)((2 * (kcx) + kk_) * RB + rb0 + mb_)) * 64 + lane];
#define GEMM_STORE_W(buf, src)                                               \
  _Pragma("unroll") for (int r_ = 0; r_ < NL; ++r_) sm.w[buf][r_ * NT + tid] = src[r_];
#define GEMM_COMPUTE(buf, ar)                                                \
  _Pragma("unroll") for (int kk_ = 0; kk_ < 2; ++kk_)                        \
    _Pragma("unroll") for (int nb_ = 0; nb_ < 8; ++nb_) {                    \
      const u32x4 bf_ = sm.w[buf][(kk_ * 8 + nb_) * 64 + lane];              \
      _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                    \
        acc[mb_][nb_] = mfma16(ar[kk_ * 4 + mb_], bf_, acc[mb_][nb_]);       \
    }

// Grid: a.grid workgroups = a.mtiles row tiles (of 256 rows) x G column
// workgroups. The row tiles of one column workgroup sit on the same XCD and
// stream the same weight chunks at the same time, so the second read hits L2.
template <int EPI, int WAVES>
__global__ __launch_bounds__(WAVES * 64, 1) void gemm_kernel(GemmArgs a) {
  constexpr int NT = WAVES * 64;
  constexpr int NL = 1024 / NT;  // 16-byte weight loads per thread per chunk
  __shared__ __attribute__((aligned(16))) Smem<WAVES> sm;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int MT = a.mtiles;
  const int G = a.grid / MT;
  // Hardware places workgroup b on XCD b % 8. Logical index q = (xcd, slot):
  // each XCD gets a contiguous piece of the iteration range.
  const int b = blockIdx.x;
  const int q = (a.grid % 8 == 0) ? (b & 7) * (a.grid >> 3) + (b >> 3) : b;
  const int mt = q % MT, g = q / MT;
  const int KC = a.KC;
  const int64_t I = (int64_t)a.tiles * KC;
  const int64_t it0 = sk_start(g, I, G), it1 = sk_start(g + 1, I, G);
  const int RB = a.Mp >> 4;
  const int rb0 = mt * 16 + wv * 4;      // first 16-row block of this wavefront
  const int row0 = mt * 256 + wv * 64;   // first row of this wavefront
  const u32x4* __restrict__ W = (const u32x4*)a.W;
  const u32x4* __restrict__ A = (const u32x4*)a.A;

  int64_t it = it0;
  bool first_seg = true;
  while (it < it1) {
    const int tile = (int)(it / KC);
    const int kc0 = (int)(it % KC);
    const int64_t tile_end = (int64_t)(tile + 1) * KC;
    const int nk = (int)((it1 < tile_end ? it1 : tile_end) - it);

    f32x4 acc[4][8];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // weights run two chunks ahead (w0 / w1), activations one chunk ahead
    u32x4 w0[NL], w1[NL], a0[8], a1[8];
    GEMM_LOAD_W(w0, it);
    if (nk > 1) { GEMM_LOAD_W(w1, it + 1); }
    GEMM_LOAD_A(a0, kc0);
    for (int s = 0;;) {
      GEMM_STORE_W(0, w0);
      __syncthreads();
      if (s + 2 < nk) { GEMM_LOAD_W(w0, it + s + 2); }
      if (s + 1 < nk) { GEMM_LOAD_A(a1, kc0 + s + 1); }
      GEMM_COMPUTE(0, a0);
      if (++s >= nk) break;
      GEMM_STORE_W(1, w1);
      __syncthreads();
      if (s + 2 < nk) { GEMM_LOAD_W(w1, it + s + 2); }
      if (s + 1 < nk) { GEMM_LOAD_A(a0, kc0 + s + 1); }
      GEMM_COMPUTE(1, a1);
      if (++s >= nk) break;
    }

    const bool whole = (kc0 == 0) && (nk == KC);
    if (whole) {
      epilogue<EPI, WAVES>(a, acc, tile, row0, wv, lane, sm);
    } else {
      // partial tile: publish, and let the last contributor finish it
      const int slot = (2 * g + (first_seg ? 0 : 1)) * MT + mt;
      f32x4* part = (f32x4*)a.partials + ((int64_t)slot * WAVES + wv) * 32 * 64;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) part[(mb * 8 + nb) * 64 + lane] = acc[mb][nb];
      const int g_lo = sk_owner((int64_t)tile * KC, I, G);
      const int g_hi = sk_owner(tile_end - 1, I, G);
      const int ncontrib = g_hi - g_lo + 1;
      __threadfence();
      __syncthreads();
      if (tid == 0) {
        const int old = atomicAdd(&a.counters[tile * MT + mt], 1);
        sm.flag = (old == ncontrib - 1);
      }
      __syncthreads();
      if (sm.flag) {
        __threadfence();
        // sum the contributors in workgroup order, one 16-row block at a time
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          f32x4 t[8];
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) t[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
          for (int gc = g_lo; gc <= g_hi; ++gc) {
            const int sl =
                (gc == g_lo && sk_start(gc, I, G) < (int64_t)tile * KC) ? 2 * gc + 1 : 2 * gc;
            const f32x4* p =
                (const f32x4*)a.partials + ((int64_t)(sl * MT + mt) * WAVES + wv) * 32 * 64;
#pragma unroll
            for (int nb = 0; nb < 8; ++nb) t[nb] += p[(mb * 8 + nb) * 64 + lane];
          }
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) acc[mb][nb] = t[nb];
        }
        epilogue<EPI, WAVES>(a, acc, tile, row0, wv, lane, sm);
        if (tid == 0) atomicExch(&a.counters[tile * MT + mt], 0);
      }
    }
    __syncthreads();
    it += nk;
    first_seg = false;
  }
}

template <int EPI>
hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  const int waves = a.Mp >= 256 ? 4 : a.Mp / 64;
  switch (waves) {
    case 1: hipLaunchKernelGGL((gemm_kernel<EPI, 1>), dim3(a.grid), dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<EPI, 2>), dim3(a.grid), dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<EPI, 4>), dim3(a.grid), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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

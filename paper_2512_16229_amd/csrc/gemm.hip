// Weight-streaming bf16 GEMM for the skinny row counts of the verify step
// (M = branches x block rows, at most a few hundred) with fused epilogues:
//   EPI_QKV    bias + rotate-half RoPE on q/k, q -> attention input, k/v -> the
//              branch K/V staging (the Pre-Write of Sec. 3.4); always in the
//              fix-up kernel, where a thread sees both RoPE halves of a column
//   EPI_RESID  residual add into the fp32 residual stream (O-proj, down-proj)
//   EPI_SWIGLU silu(gate) * up -> packed bf16 operand of the down projection
//   EPI_LMHEAD per (row, column tile) softmax statistics: max, argmax, sum of
//              exp (the logits never reach memory)
//
// Work decomposition. The weight is a sequence of 16-column blocks; a column
// tile is NB consecutive blocks. A workgroup (4 wavefronts, one per 64 rows)
// covers one 256-row tile, so each weight byte crosses HBM once per row tile,
// and one (column tile, k-split): with Q quads of k-chunks, split s owns
// [s Q / S, (s + 1) Q / S). The tile width NB and the split count S are chosen
// per GEMM on the host:
//   S == 1  whole K in one workgroup, epilogue in place (no partial sums);
//   S  > 1  fp32 partial sums, added in split order (deterministic): for the
//           residual projections by the RMSNorm kernel that follows them, for
//           QKV by gemm_fixup_kernel, which also runs the QKV epilogue (QKV
//           always takes this path).
//
// Pipeline. One iteration is a 64-wide k-chunk of one tile. Its NB x 2 KiB of
// weights go global -> LDS directly (global_load_lds, no registers) into a
// 6-slot ring, and each wavefront's 8 activation fragments (L2-resident) into
// one of 4 register sets; both are issued 4 iterations ahead. K is padded to a
// multiple of 256, so a tile always spans a multiple of 4 iterations and the
// register set of iteration j is the static j % 4: the loop is unrolled by 4
// and no register set is ever rotated. Vector memory operations complete in
// issue order, so "iterations j, j + 1 have landed" is one vmcnt wait on the
// number of operations issued after them; one workgroup barrier per pair of
// iterations.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace {

constexpr int GEMM_THREADS = 256;
constexpr int LEAD = 4;         // iterations between issue and use (= activation register sets)
constexpr int RING = LEAD + 2;  // weight chunks in LDS: a pair in use + LEAD in flight

template <int EPI, int NB>
struct GemmSmem {
  static constexpr int CHUNK = NB * 2048;  // bytes of weights per iteration
  static constexpr int BYTES = RING * CHUNK;
  static_assert(EPI != EPI_LMHEAD || 4 * 64 * 16 * 12 <= RING * CHUNK, "reduction area fits");
};

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Asynchronous global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane l copies base + voff(l) to bytes [16 l, 16 l + 16) of the 1 KiB LDS block
// at lds_addr (wave-uniform, passed in M0). base is wave-uniform (SGPRs), so
// the only per-lane address is the constant voff = 16 lane. The compiler does
// not track the copy: completion is awaited with an explicit vmcnt wait
// before the workgroup barrier. NT selects the nontemporal (streaming) cache
// policy: measured per projection, it raises the sustained rate of the long
// gate/up weight stream (about 7 %) but slows the short ones (QKV, O, down)
// and the LM head, which keep the default policy.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  // the "s" constraint alone does not keep a value the compiler thinks may
  // diverge out of VGPRs: make the scalar copy explicit
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const void*)(((uint64_t)hi << 32) | lo);
}
template <bool NT>
__device__ __forceinline__ void lds_dma16(const void* base, uint32_t voff, uint32_t lds_addr) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                 ::"s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(uniform_ptr(base))
                 : "memory");
  else
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 ::"s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(uniform_ptr(base))
                 : "memory");
}

// Four activation fragments (1 KiB apart) at a wave-uniform base -> registers.
// Issued as inline assembly so that, like the LDS copies, the compiler does not
// track them: its own waits would count only the loads it knows of and so
// stall on younger loads. Nothing reads the registers before the explicit
// vmcnt wait of the iteration that uses them; pin_landed() then hands them to
// the compiler.
__device__ __forceinline__ void load_frag4(u32x4& d0, u32x4& d1, u32x4& d2, u32x4& d3,
                                           const void* base, uint32_t voff) {
  asm volatile(
      "global_load_dwordx4 %0, %4, %5\n\t"
      "global_load_dwordx4 %1, %4, %5 offset:1024\n\t"
      "global_load_dwordx4 %2, %4, %5 offset:2048\n\t"
      "global_load_dwordx4 %3, %4, %5 offset:3072"
      : "=&v"(d0), "=&v"(d1), "=&v"(d2), "=&v"(d3)
      : "v"(voff), "s"(uniform_ptr(base))
      : "memory");
}
__device__ __forceinline__ void pin_landed(u32x4& v) { asm volatile("" : "+v"(v)); }
// After the loop the last iterations' loads (repeats of the last chunk) are
// still in flight into the activation registers: wait for them, and keep the
// registers alive until then so that nothing else is placed in them earlier.
#define GEMM_DRAIN()                                                                     \
  {                                                                                      \
    wait_vmcnt<0>();                                                                     \
    _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                   \
      pin_landed(a0[i_]);                                                                \
      pin_landed(a1[i_]);                                                                \
      pin_landed(a2[i_]);                                                                \
      pin_landed(a3[i_]);                                                                \
    }                                                                                    \
  }

// c += a^T b on a 16x16x32 bf16 tile, accumulating in place in AGPRs. Written as
// inline assembly with a tied operand: with the builtin the register allocator
// renames accumulators between the unrolled iterations and then copies them
// back at the loop edge. The compiler does not see these as MFMAs, so the
// hazard wait states are explicit: mfma_settle() before accumulators are read
// or rewritten by other instructions, and after they are zeroed.
__device__ __forceinline__ void mfma_acc(f32x4& c, const u32x4& a, const u32x4& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
// FP8 (E4M3 x E4M3) form: one 16x16x128 MFMA over 32 bytes per lane of each
// operand, both operands in the default E4M3 format, unscaled (the real scales
// are applied in the epilogue; the block-scaled form with unit scales measured
// 0.3 % slower over the FP8 step). A lane's byte b of A and byte b of B meet in
// the same product, so any placement of K inside the 32 bytes works as long as
// A and W use the same.
__device__ __forceinline__ void mfma_acc_f8(f32x4& c, const u32x8& a, const u32x8& b) {
  asm volatile("v_mfma_f32_16x16x128_f8f6f4 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
__device__ __forceinline__ u32x8 cat8(const u32x4& lo, const u32x4& hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ __forceinline__ void mfma_settle() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// ------------------------------------------------------------------ epilogues
// acc[mb][nb][j]: row row0 + 16 mb + 4 g + j, column 16 (tile NB + nb) + c16
// of this wavefront (g = lane / 16, c16 = lane % 16); the SwiGLU GEMM holds
// the transposed tile (see swiglu_epilogue).

// FP8: the accumulated products times the row's and the column's scales
// (acc[mb][nb][j]: row row0 + 16 mb + 4 g + j, packed column 16 (tile NB + nb) + c16)
template <int NB>
__device__ __forceinline__ void f8_scale(const GemmArgs& a, f32x4 (&acc)[4][NB], int tile,
                                         int row0, int lane) {
  const int g = lane >> 4, c16 = lane & 15;
  float swc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) swc[nb] = a.sw[(tile * NB + nb) * 16 + c16];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float sr = a.sa[row0 + mb * 16 + g * 4 + j];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb][j] = acc[mb][nb][j] * sr * swc[nb];
    }
}

template <int NB>
__device__ __forceinline__ void resid_epilogue(const GemmArgs& a, f32x4 (&acc)[4][NB], int tile,
                                               int row0, int lane) {
  const int g = lane >> 4, c16 = lane & 15;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = row0 + mb * 16 + g * 4 + j;
      if (r >= a.M) continue;
      float* xr = a.x + (int64_t)r * a.N;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int n = (tile * NB + nb) * 16 + c16;
        if (n < a.N) xr[n] += acc[mb][nb][j];
      }
    }
}

// gate / up blocks alternate (block 2p: gate columns 16p.., block 2p + 1: up);
// output block p of the tile -> columns 16 (tile NB / 2 + p) of the packed
// down-projection operand. The SwiGLU GEMM accumulates the transposed tile
// (weights as the MFMA's first operand), so acc[mb][nb][j] holds row
// row0 + 16 mb + c16, column 16 (tile NB + nb) + 4 g + j: a lane's four
// outputs of a block are four consecutive columns of one row. The packed
// operand keeps 8 consecutive columns of a row in one 16-byte lane slot, so
// lanes l and l ^ 16 (column groups 4g and 4(g ^ 1) of the same row) trade
// halves with one permlane swap per dword: afterwards the even lane holds the
// slot of row block mb, the odd lane the slot of row block mb + 1, and each
// writes 16 bytes.
template <int NB, bool F8>
__device__ __forceinline__ void swiglu_epilogue(const GemmArgs& a, f32x4 (&acc)[4][NB], int tile,
                                                int row0, int lane) {
  constexpr int PAIRS = NB / 2;
  const int g = lane >> 4, c16 = lane & 15;
  const int Nout = a.N >> 1;
  float mxr[4] = {0.f, 0.f, 0.f, 0.f};  // FP8: largest |output| of each row block's row
  auto swiglu4 = [&](int mb, int p, uint32_t (&hv)[2]) {
    // FP8: scales of the row (this lane's) and of the gate / up columns
    const float sr = F8 ? a.sa[row0 + mb * 16 + c16] : 1.f;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      float h2[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int j = 2 * jj + u;
        float gt = acc[mb][2 * p][j], up = acc[mb][2 * p + 1][j];
        if constexpr (F8) {
          gt = gt * sr * a.sw[(tile * NB + 2 * p) * 16 + 4 * g + j];
          up = up * sr * a.sw[(tile * NB + 2 * p + 1) * 16 + 4 * g + j];
        }
        // silu(g) = g / (1 + e^-g) with the hardware exp2 and reciprocal (about
        // 1 ulp each, far below the bf16 rounding of the result)
        const float ex = __builtin_amdgcn_exp2f(-gt * 1.4426950408889634f);
        h2[u] = gt * __builtin_amdgcn_rcpf(1.0f + ex) * up;
      }
      hv[jj] = (uint32_t)f2bf_bits(h2[0]) | ((uint32_t)f2bf_bits(h2[1]) << 16);
      if constexpr (F8)
        mxr[mb] = fmaxf(mxr[mb], fmaxf(fabsf(bf2f_bits(hv[jj] & 0xffffu)), fabsf(bf2f_bits(hv[jj] >> 16))));
    }
  };
#pragma unroll
  for (int mp = 0; mp < 2; ++mp) {
    const int r = row0 + (2 * mp + (g & 1)) * 16 + c16;
#pragma unroll
    for (int p = 0; p < PAIRS; ++p) {
      uint32_t h0[2], h1[2];
      swiglu4(2 * mp, p, h0);
      swiglu4(2 * mp + 1, p, h1);
      const auto w0 = __builtin_amdgcn_permlane16_swap(h0[0], h1[0], false, false);
      const auto w1 = __builtin_amdgcn_permlane16_swap(h0[1], h1[1], false, false);
      const int col = (tile * PAIRS + p) * 16 + (g >> 1) * 8;
      if (r < a.M && col < Nout)
        *(uint4*)(a.a_out + packA_off(r, col, a.Mp)) = make_uint4(w0[0], w1[0], w0[1], w1[1]);
    }
  }
  if constexpr (F8) {
    // the row maxima of this tile's outputs (the stored bf16 values) into the
    // per-row maximum over all tiles: the lanes c16 + 16 g hold the same row;
    // an unsigned maximum of the bits orders non-negative floats exactly
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      float m = fmaxf(mxr[mb], __shfl_xor(mxr[mb], 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      const int r = row0 + mb * 16 + c16;
      if (g == 0 && r < a.M) atomicMax(a.rowmax + r, __float_as_uint(m));
    }
  }
}

// per-row (max, argmax, sum exp(l - max)) over this tile's valid columns
// (column < vocab, column != mask token) -> pm / ps / pi [row][tile]. Each lane
// first reduces its NB columns of each of its 16 rows; the 16 lane partials of
// a row then meet in LDS (red: this wavefront's 64 x 16 x 3 words) and one lane
// per row merges them in column order (ties: lowest column).
template <int NB>
__device__ __forceinline__ void lm_epilogue(const GemmArgs& a, f32x4 (&acc)[4][NB], int tile,
                                            int row0, int lane, float* red) {
  constexpr float LOG2E = 1.4426950408889634f;
  const int g = lane >> 4, c16 = lane & 15;
  float* rm = red;
  float* rs = red + 64 * 16;
  int* ri = (int*)(red + 2 * 64 * 16);
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float m = -INFINITY;
      int mi = 0x7fffffff;
      float v[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = (tile * NB + nb) * 16 + c16;
        v[nb] = (col < a.vocab && col != a.mask_id) ? acc[mb][nb][j] : -INFINITY;
        mi = v[nb] > m ? col : mi;  // strict: the lowest column of equal maxima
        m = fmaxf(m, v[nb]);
      }
      float s = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) s += __builtin_amdgcn_exp2f((v[nb] - m) * LOG2E);
      if (m == -INFINITY) s = 0.f;
      const int o = (mb * 16 + g * 4 + j) * 16 + c16;
      rm[o] = m;
      rs[o] = s;
      ri[o] = mi;
    }
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wavefront's LDS writes done
  __builtin_amdgcn_wave_barrier();
  float M = -INFINITY, S = 0.f;
  int I = 0x7fffffff;
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const float mc = rm[lane * 16 + c], sc = rs[lane * 16 + c];
    const int ic = ri[lane * 16 + c];
    if (mc > M) {
      S = S * __builtin_amdgcn_exp2f((M - mc) * LOG2E) + sc;
      M = mc;
      I = ic;
    } else if (mc == M) {
      S += sc;
      I = ic < I ? ic : I;
    } else {
      S += sc * __builtin_amdgcn_exp2f((mc - M) * LOG2E);
    }
  }
  const int r = row0 + lane;
  if (r < a.M) {
    const int64_t o = (int64_t)r * a.tiles + tile;
    a.pm[o] = M;
    a.ps[o] = M == -INFINITY ? 0.f : S;
    a.pi[o] = I;
  }
}

// ------------------------------------------------------------------ main loop
// Loads of one iteration: 8 activation fragments into register set `set` (two
// groups of 4, k-halves 0 and 1) and the NB x 2 KiB weight chunk into ring
// slot `slot` (NB / 2 copies of 1 KiB per wavefront). Weight layout
// [tile][KC][NB][2][64 lanes][8]: the chunk of iteration (tile, kc) is one
// contiguous run, and so is a tile's whole k-range. The addresses advance by
// one k-chunk per issued iteration (a_next, w_next), from kc0 to the end of the
// range and then from its start (rotation, GemmArgs::rot); after the last of
// the range's iterations the last chunk is issued again (an L2 hit), which keeps
// every wait count constant and the loop branch-free.
#define GEMM_ISSUE_A(set, half)                                                          \
  load_frag4(set[4 * (half) + 0], set[4 * (half) + 1], set[4 * (half) + 2],              \
             set[4 * (half) + 3], a_next + (half) * a_half, voff)
#define GEMM_ISSUE_W(r, slot)                                                            \
  lds_dma16<EPI == EPI_SWIGLU>(w_next + (r) * 4096, voff,                              \
            lds_wave + (uint32_t)(slot) * (uint32_t)SM::CHUNK + (uint32_t)(r) * 4096u)
#define GEMM_ADVANCE_LOAD()                                                              \
  {                                                                                      \
    if (li + 1 < n_it) {                                                                 \
      ++li;                                                                              \
      if (lk + 1 < kc_end) {                                                             \
        ++lk;                                                                            \
        a_next += a_kstep;                                                               \
        w_next += SM::CHUNK;                                                             \
      } else {                                                                           \
        lk = kc_beg;                                                                     \
        a_next -= (int64_t)(n_it - 1) * a_kstep;                                         \
        w_next -= (int64_t)(n_it - 1) * SM::CHUNK;                                       \
      }                                                                                  \
    }                                                                                    \
  }
#define GEMM_ISSUE(set, slot)                                                            \
  {                                                                                      \
    GEMM_ISSUE_A(set, 0);                                                                \
    GEMM_ISSUE_A(set, 1);                                                                \
    _Pragma("unroll") for (int r_ = 0; r_ < NB / 2; ++r_) GEMM_ISSUE_W(r_, slot);        \
    GEMM_ADVANCE_LOAD();                                                                 \
  }

// Two iterations j, j + 1 per workgroup barrier. Their 4 NB weight fragments
// are read from LDS BPF fragments ahead of the MFMAs that use them (across
// the iteration boundary); the loads of iterations j + 4 and j + 5 are spread
// over the MFMA stream (an activation half once the MFMAs reading it have
// issued, the weight copies from the second fragment of each iteration on).
// Scheduling barriers keep this order. Every iteration issues exactly OPS
// operations, so "j and j + 1 have landed" is vmcnt(2 OPS); the slots written
// here held iterations j - 2 and j - 1, which every wavefront finished before
// this barrier.
constexpr int BPF = 4;
#define GEMM_PAIR(s0, s1)                                                                \
  {                                                                                      \
    wait_vmcnt<2 * OPS>();                                                               \
    lds_barrier();                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                   \
      pin_landed(s0[i_]);                                                                \
      pin_landed(s1[i_]);                                                                \
    }                                                                                    \
    const u32x4* wl0_ = (const u32x4*)(smem + cs * SM::CHUNK);                           \
    const int c1_ = cs + 1 == RING ? 0 : cs + 1;                                         \
    const u32x4* wl1_ = (const u32x4*)(smem + c1_ * SM::CHUNK);                          \
    const int is0_ = cs >= 2 ? cs - 2 : cs + RING - 2; /* slot of iteration j - 2 */    \
    const int is1_ = is0_ + 1 == RING ? 0 : is0_ + 1;                                    \
    u32x4 bf_[4 * NB];                                                                   \
    _Pragma("unroll") for (int f_ = 0; f_ < BPF; ++f_)                                   \
      bf_[f_] = wl0_[((f_ % NB) * 2 + f_ / NB) * 64 + lane];                             \
    __builtin_amdgcn_sched_barrier(0);                                                   \
    _Pragma("unroll") for (int f_ = 0; f_ < 4 * NB; ++f_) {                              \
      const int e_ = f_ / (2 * NB), g_ = f_ % (2 * NB); /* iteration, fragment */        \
      if (f_ + BPF < 4 * NB) {                                                           \
        const int fn_ = f_ + BPF, gn_ = fn_ % (2 * NB);                                  \
        bf_[fn_] = (fn_ < 2 * NB ? wl0_ : wl1_)[((gn_ % NB) * 2 + gn_ / NB) * 64 + lane];  \
      }                                                                                  \
      _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_)                                \
        if constexpr (EPI == EPI_SWIGLU) /* transposed tile: lanes hold output rows */  \
          mfma_acc(acc[mb_][g_ % NB], bf_[f_], (e_ ? s1 : s0)[(g_ / NB) * 4 + mb_]);     \
        else                                                                             \
          mfma_acc(acc[mb_][g_ % NB], (e_ ? s1 : s0)[(g_ / NB) * 4 + mb_], bf_[f_]);     \
      if (g_ >= 1 && g_ <= NB / 2) GEMM_ISSUE_W(g_ - 1, e_ ? is1_ : is0_);               \
      if (g_ == NB - 1) GEMM_ISSUE_A((e_ ? s1 : s0), 0);                                 \
      if (g_ == 2 * NB - 1) {                                                            \
        GEMM_ISSUE_A((e_ ? s1 : s0), 1);                                                 \
        GEMM_ADVANCE_LOAD();                                                             \
      }                                                                                  \
      __builtin_amdgcn_sched_barrier(0);                                                 \
    }                                                                                    \
    cs = cs + 2 >= RING ? cs + 2 - RING : cs + 2;                                        \
  }

// FP8 form of GEMM_PAIR: a weight unit (block, k-half) covers 64 values of K
// (16 per lane), and the units are read in (block, half) order, so both halves
// of a block are in registers together; each block then takes one 16x16x128 MFMA per
// row block with both activation halves as its first operand. The activation
// set of an iteration is read until its last block, so both halves are
// reissued at the end of the iteration (the weight copies as in GEMM_PAIR).
#define GEMM_PAIR_F8(s0, s1)                                                             \
  {                                                                                      \
    wait_vmcnt<2 * OPS>();                                                               \
    lds_barrier();                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                   \
      pin_landed(s0[i_]);                                                                \
      pin_landed(s1[i_]);                                                                \
    }                                                                                    \
    const u32x4* wl0_ = (const u32x4*)(smem + cs * SM::CHUNK);                           \
    const int c1_ = cs + 1 == RING ? 0 : cs + 1;                                         \
    const u32x4* wl1_ = (const u32x4*)(smem + c1_ * SM::CHUNK);                          \
    const int is0_ = cs >= 2 ? cs - 2 : cs + RING - 2;                                   \
    const int is1_ = is0_ + 1 == RING ? 0 : is0_ + 1;                                    \
    u32x4 bf_[4 * NB];                                                                   \
    _Pragma("unroll") for (int f_ = 0; f_ < BPF; ++f_) bf_[f_] = wl0_[f_ * 64 + lane];    \
    __builtin_amdgcn_sched_barrier(0);                                                   \
    _Pragma("unroll") for (int f_ = 0; f_ < 4 * NB; ++f_) {                              \
      const int e_ = f_ / (2 * NB), g_ = f_ % (2 * NB); /* iteration, unit */           \
      if (f_ + BPF < 4 * NB) {                                                           \
        const int fn_ = f_ + BPF, gn_ = fn_ % (2 * NB);                                  \
        bf_[fn_] = (fn_ < 2 * NB ? wl0_ : wl1_)[gn_ * 64 + lane];                        \
      }                                                                                  \
      if (g_ & 1) {                                                                      \
        const u32x8 b8_ = cat8(bf_[f_ - 1], bf_[f_]);                                    \
        _Pragma("unroll") for (int mb_ = 0; mb_ < 4; ++mb_) {                            \
          const u32x8 a8_ = cat8((e_ ? s1 : s0)[mb_], (e_ ? s1 : s0)[4 + mb_]);          \
          if constexpr (EPI == EPI_SWIGLU)                                               \
            mfma_acc_f8(acc[mb_][g_ >> 1], b8_, a8_);                                    \
          else                                                                           \
            mfma_acc_f8(acc[mb_][g_ >> 1], a8_, b8_);                                    \
        }                                                                                \
      }                                                                                  \
      if (g_ >= 1 && g_ <= NB / 2) GEMM_ISSUE_W(g_ - 1, e_ ? is1_ : is0_);               \
      if (g_ == 2 * NB - 1) {                                                            \
        GEMM_ISSUE_A((e_ ? s1 : s0), 0);                                                 \
        GEMM_ISSUE_A((e_ ? s1 : s0), 1);                                                 \
        GEMM_ADVANCE_LOAD();                                                             \
      }                                                                                  \
      __builtin_amdgcn_sched_barrier(0);                                                 \
    }                                                                                    \
    cs = cs + 2 >= RING ? cs + 2 - RING : cs + 2;                                        \
  }

template <int EPI, int NB, bool F8>
__global__ __launch_bounds__(GEMM_THREADS, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_kernel(GemmArgs a) {
  using SM = GemmSmem<EPI, NB>;
  // FP8: the epilogues of RESID and LMHEAD take scaled sums (f8_scale), SWIGLU
  // scales inside its epilogue, QKV in the fix-up (its partial sums are raw)
  constexpr int OPS = 8 + NB / 2;  // vector memory operations per wavefront per iteration
  static_assert(NB % 2 == 0 && 3 * OPS <= 63, "tile width");
  static_assert(RING == 6 && LEAD == 4, "pair schedule");
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t sW_base = (uint32_t)(uintptr_t)smem;

  // Hardware places workgroup b on XCD b % 8; the remap gives each XCD a
  // contiguous range of q (XCD x: grid / 8 workgroups, one more when x <
  // grid % 8), so the row tiles of one column workgroup (adjacent q) share an
  // L2 and read each weight chunk from HBM once.
  const int b = blockIdx.x, grid = gridDim.x;
  const int xcd = b & 7, g8 = grid >> 3, g8r = grid & 7;
  const int q = xcd * g8 + (xcd < g8r ? xcd : g8r) + (b >> 3);
  const int MT = a.mtiles;
  const int mt = q % MT, c = q / MT;
  const int KC = a.KC, QT = KC >> 2;
  // workgroup c of a row tile: k-split c / T, column tile c % T. Split-major, so
  // that the workgroups of one XCD (consecutive q) share a k-range and with it
  // the slice of the activation operand they stream: it stays in that XCD's
  // L2 instead of being fetched once per column tile.
  const int split = c / a.tiles;
  const int t_lo = c % a.tiles;
  const int kc_beg = 4 * (split * QT / a.splits);
  const int kc_end = 4 * ((split + 1) * QT / a.splits);
  if (t_lo >= a.tiles || kc_beg >= kc_end) return;
  const int nq = (kc_end - kc_beg) >> 2;  // quads of iterations per tile
  const int RB = a.Mp >> 4;
  const int rb0 = mt * 16 + wv * 4;     // first 16-row block of this wavefront
  const int row0 = mt * 256 + wv * 64;  // first row of this wavefront
  const uint32_t voff = (uint32_t)lane * 16u;
  // activation fragment (kb, rb) at A + ((kb RB) + rb) KiB: k-chunk kc, half h
  // of this wavefront's first row block -> a_next + h a_half
  const int64_t a_half = (int64_t)RB * 1024, a_kstep = 2 * a_half;
  const int n_it = kc_end - kc_beg;  // iterations of this workgroup
  const int kc0 = kc_beg + (a.rot ? 4 * (t_lo % nq) : 0);  // first k-chunk
  const char* a_next = (const char*)a.A + ((int64_t)2 * kc0 * RB + rb0) * 1024;
  // weight chunk (tile, kc) at W + (tile KC + kc) CHUNK; its 1 KiB unit u (block
  // u / 2, k-half u % 2) at + u KiB; wavefront wv copies units 4 r + wv
  const char* w_next = (const char*)a.W + ((int64_t)t_lo * KC + kc0) * SM::CHUNK + wv * 1024;
  const uint32_t lds_wave = sW_base + (uint32_t)wv * 1024u;
  int lk = kc0;  // k-chunk of the next iteration to issue
  int li = 0;    // iterations issued before it

  f32x4 acc[4][NB];
  u32x4 a0[8], a1[8], a2[8], a3[8];
  GEMM_ISSUE(a0, 0);
  GEMM_ISSUE(a1, 1);
  GEMM_ISSUE(a2, 2);
  GEMM_ISSUE(a3, 3);
  int cs = 0;  // ring slot of the current iteration

  {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    mfma_settle();
    for (int qq = 0; qq < nq; ++qq) {
      if constexpr (F8) {
        GEMM_PAIR_F8(a0, a1);
        GEMM_PAIR_F8(a2, a3);
      } else {
        GEMM_PAIR(a0, a1);
        GEMM_PAIR(a2, a3);
      }
    }
    GEMM_DRAIN();
    mfma_settle();
    if constexpr (F8 && (EPI == EPI_RESID || EPI == EPI_LMHEAD)) f8_scale<NB>(a, acc, t_lo, row0, lane);
    if (EPI != EPI_QKV && a.splits == 1) {
      if constexpr (EPI == EPI_LMHEAD) {
        lds_barrier();  // the ring becomes the reduction area (every copy has landed)
        lm_epilogue<NB>(a, acc, t_lo, row0, lane, (float*)smem + wv * 64 * 16 * 3);
      }
      if constexpr (EPI == EPI_RESID) resid_epilogue<NB>(a, acc, t_lo, row0, lane);
      if constexpr (EPI == EPI_SWIGLU) swiglu_epilogue<NB, F8>(a, acc, t_lo, row0, lane);
    } else if constexpr (EPI == EPI_RESID) {
      // row-major partial sums [split][Mp][N], added by the following RMSNorm
      const int g = lane >> 4, c16 = lane & 15;
      float* part = a.partials + (int64_t)split * a.Mp * a.N;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float* pr = part + (int64_t)(row0 + mb * 16 + g * 4 + j) * a.N;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const int n = (t_lo * NB + nb) * 16 + c16;
            if (n < a.N) pr[n] = acc[mb][nb][j];
          }
        }
    } else {
      const int64_t slot = ((int64_t)mt * a.tiles + t_lo) * a.splits + split;
      f32x4* part = (f32x4*)a.partials + (slot * 4 + wv) * 4 * NB * 64;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) part[(mb * NB + nb) * 64 + lane] = acc[mb][nb];
    }
  }
  wait_vmcnt<0>();  // nothing may still be writing LDS when the workgroup ends
}

// QKV: sum the S partials of one f32x4 of the output (4 rows, 1 column) in
// split order and run the epilogue. One thread per (row tile, column tile, wave,
// 16-row block, 16-column block, lane): the same indexing as gemm_kernel's
// partial store, so each warp-wide load is 1 KiB contiguous. The split count SC
// (1..8, QKV_MAX_SPLITS) is a constant, so that every load of a thread (the
// split sums of its column and of its rotation partner, the rotary rows, bias
// and scales) is in flight before the first add.
template <int EPI, int NB, int SC>
__global__ __launch_bounds__(256) void gemm_fixup_kernel(GemmArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int lane = (int)(gid & 63);
  int64_t rest = gid >> 6;
  const int nb = (int)(rest % NB);
  rest /= NB;
  const int mb = (int)(rest & 3);
  rest >>= 2;
  const int wv = (int)(rest & 3);
  rest >>= 2;
  const int tile = (int)(rest % a.tiles);
  const int mt = (int)(rest / a.tiles);
  if (mt >= a.mtiles) return;
  const int g = lane >> 4, c16 = lane & 15;
  const int r0 = mt * 256 + wv * 64 + mb * 16 + g * 4;
  const int n = (tile * NB + nb) * 16 + c16;
  if (n >= a.N || r0 >= a.M) return;
  const int D = a.d, HD = D >> 1;
  const int qcols = a.Hq * D, kcols = a.Hkv * D;
  const int sect = n < qcols ? 0 : (n < qcols + kcols ? 1 : 2);
  const int base = sect == 0 ? 0 : (sect == 1 ? qcols : qcols + kcols);
  const int head = (n - base) / D, dim = (n - base) % D;
  if (sect < 2 && dim >= HD) return;  // written with its rotation partner
  const bool rot = sect < 2;
  const int n2 = rot ? n + HD : n;  // the partner column (V: the column itself, unused)
  const int64_t sstride = (int64_t)4 * 4 * NB * 64;  // f32x4 between consecutive splits
  auto first = [&](int col) {
    const int t2 = (col >> 4) / NB, nb2 = (col >> 4) % NB;
    return (const f32x4*)a.partials +
           ((((int64_t)mt * a.tiles + t2) * a.splits * 4 + wv) * 4 * NB + mb * NB + nb2) * 64 + lane;
  };
  const f32x4* p1 = first(n);
  const f32x4* p2 = first(n2);
  f32x4 v1 = p1[0], v2 = p2[0];
#pragma unroll
  for (int s = 1; s < SC; ++s) {
    v1 += p1[s * sstride];
    v2 += p2[s * sstride];
  }
  // rows r0 .. r0 + 3 (those past M read row M - 1's table entries and are not stored)
  int br[4], pos[4];
  float2 cs[4];
  float sr[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = r0 + j < a.M ? r0 + j : a.M - 1;
    br[j] = r / a.L;
    pos[j] = r % a.L;
    cs[j] = rot ? *(const float2*)(a.rope + ((int64_t)(a.P + pos[j]) * HD + dim) * 2)
                : make_float2(1.f, 0.f);
    sr[j] = a.f8 && r0 + j < a.M ? a.sa[r0 + j] : 0.f;
  }
  const float b1 = a.bias ? a.bias[n] : 0.f;
  const float b2 = (a.bias && rot) ? a.bias[n2] : 0.f;
  const float sw1 = a.f8 ? a.sw[n] : 0.f, sw2 = a.f8 && rot ? a.sw[n2] : 0.f;
  if (a.f8) {  // FP8 operands: the sums of products times the row and column scales
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v1[j] = v1[j] * sr[j] * sw1;
      if (rot) v2[j] = v2[j] * sr[j] * sw2;
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (r0 + j >= a.M) continue;
    const int i = pos[j];
    float o1 = v1[j] + b1, o2 = 0.f;
    if (rot) {
      const float x1 = o1, x2 = v2[j] + b2;
      o1 = x1 * cs[j].x - x2 * cs[j].y;
      o2 = x2 * cs[j].x + x1 * cs[j].y;
    }
    if (sect == 0) {
      uint16_t* qo = a.q_out + (((int64_t)br[j] * a.Hq + head) * a.L + i) * D;
      qo[dim] = f2bf_bits(o1);
      qo[dim + HD] = f2bf_bits(o2);
    } else {
      // staging head (K or V) of this branch and layer, in the KV tile layout
      uint16_t* st = a.staging + ((((int64_t)br[j] * a.layers + a.layer) * 2 + (sect - 1)) *
                                      a.Hkv + head) * D * a.vlds;
      if (sect == 1) {
        st[kv_k_off(i, dim, D)] = f2bf_bits(o1);
        st[kv_k_off(i, dim + HD, D)] = f2bf_bits(o2);
      } else {
        st[kv_v_off(i, dim, D)] = f2bf_bits(o1);
      }
    }
  }
}

template <int EPI, int NB, bool F8 = false>
hipError_t launch_nb(const GemmArgs& a, hipStream_t s) {
  const int grid = a.mtiles * a.gcols;
  hipLaunchKernelGGL((gemm_kernel<EPI, NB, F8>), dim3(grid), dim3(GEMM_THREADS), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if constexpr (EPI == EPI_QKV) {
    const int64_t threads = (int64_t)a.mtiles * a.tiles * 4 * 4 * NB * 64;
    const dim3 fg((unsigned)((threads + 255) / 256));
    switch (a.splits) {
#define FIXUP(SC) hipLaunchKernelGGL((gemm_fixup_kernel<EPI, NB, SC>), fg, dim3(256), 0, s, a)
      case 1: FIXUP(1); break;
      case 2: FIXUP(2); break;
      case 3: FIXUP(3); break;
      case 4: FIXUP(4); break;
      case 5: FIXUP(5); break;
      case 6: FIXUP(6); break;
      case 7: FIXUP(7); break;
      case 8: FIXUP(8); break;
      default: return hipErrorInvalidValue;  // launch_gemm admits at most QKV_MAX_SPLITS
#undef FIXUP
    }
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

int gemm_smem_bytes(int epi, int nb) {
  switch (epi * 16 + nb) {
    case EPI_QKV * 16 + 4: return GemmSmem<EPI_QKV, 4>::BYTES;
    case EPI_QKV * 16 + 8: return GemmSmem<EPI_QKV, 8>::BYTES;
    case EPI_RESID * 16 + 4: return GemmSmem<EPI_RESID, 4>::BYTES;
    case EPI_RESID * 16 + 8: return GemmSmem<EPI_RESID, 8>::BYTES;
    case EPI_SWIGLU * 16 + 10: return GemmSmem<EPI_SWIGLU, 10>::BYTES;
    case EPI_LMHEAD * 16 + 8: return GemmSmem<EPI_LMHEAD, 8>::BYTES;
    case EPI_LMHEAD * 16 + 10: return GemmSmem<EPI_LMHEAD, 10>::BYTES;
  }
  return -1;
}

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  // (epilogue, tile width) pairs the host planner may choose; splits > 1 only
  // for EPI_QKV and EPI_RESID
  if (a.splits > 1 && (epi == EPI_SWIGLU || epi == EPI_LMHEAD)) return hipErrorInvalidValue;
  if (a.KC % 4 || a.KC < 4 || a.splits < 1 || a.splits > a.KC / 4 || a.mtiles < 1 ||
      a.gcols < 1 || a.Mp != 256 * a.mtiles)
    return hipErrorInvalidValue;
  if (a.gcols != a.tiles * a.splits) return hipErrorInvalidValue;
  if (epi == EPI_QKV && a.splits > QKV_MAX_SPLITS) return hipErrorInvalidValue;
  if (a.f8) {
    if (!a.sa || !a.sw || (epi == EPI_SWIGLU && !a.rowmax)) return hipErrorInvalidValue;
    switch (epi * 16 + a.nb) {
      case EPI_QKV * 16 + 4: return launch_nb<EPI_QKV, 4, true>(a, s);
      case EPI_QKV * 16 + 8: return launch_nb<EPI_QKV, 8, true>(a, s);
      case EPI_RESID * 16 + 4: return launch_nb<EPI_RESID, 4, true>(a, s);
      case EPI_RESID * 16 + 8: return launch_nb<EPI_RESID, 8, true>(a, s);
      case EPI_SWIGLU * 16 + 10: return launch_nb<EPI_SWIGLU, 10, true>(a, s);
      case EPI_LMHEAD * 16 + 8: return launch_nb<EPI_LMHEAD, 8, true>(a, s);
      case EPI_LMHEAD * 16 + 10: return launch_nb<EPI_LMHEAD, 10, true>(a, s);
    }
    return hipErrorInvalidValue;
  }
  switch (epi * 16 + a.nb) {
    case EPI_QKV * 16 + 4: return launch_nb<EPI_QKV, 4>(a, s);
    case EPI_QKV * 16 + 8: return launch_nb<EPI_QKV, 8>(a, s);
    case EPI_RESID * 16 + 4: return launch_nb<EPI_RESID, 4>(a, s);
    case EPI_RESID * 16 + 8: return launch_nb<EPI_RESID, 8>(a, s);
    case EPI_SWIGLU * 16 + 10: return launch_nb<EPI_SWIGLU, 10>(a, s);
    case EPI_LMHEAD * 16 + 8: return launch_nb<EPI_LMHEAD, 8>(a, s);
    case EPI_LMHEAD * 16 + 10: return launch_nb<EPI_LMHEAD, 10>(a, s);
  }
  return hipErrorInvalidValue;
}

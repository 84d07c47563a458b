// The verify forward's working buffers and the internal entry that runs it on
// a given set of them (internal to liblopa; the C ABI is include/lopa.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/lopa.h"

// Device memory one verify forward writes and reads besides its inputs,
// outputs, the weights and the KV cache / staging: the residual stream, the
// packed GEMM operands, the attention queries, split-K partial sums, the LM
// head's per-tile softmax statistics, and the FP8 operands and scales.
struct VerifyWs {
  float* x = nullptr;          // [Mp][H] fp32 residual stream
  uint16_t* abuf = nullptr;    // packed [Mp][H] bf16 operand
  uint16_t* fbuf = nullptr;    // packed [Mp][round256(F)] bf16 operand (padding columns zero)
  uint16_t* qbuf = nullptr;    // [branches][Hq][L][d] bf16 queries
  float* partials = nullptr;   // split-K partial sums; the grouped attention's scratch
  size_t partials_bytes = 0;
  float* pm = nullptr;         // [Mp][LM-head tiles] max
  float* ps = nullptr;         // [Mp][LM-head tiles] sum of exp
  int32_t* pi = nullptr;       // [Mp][LM-head tiles] argmax
  uint8_t* a8_gu = nullptr;    // FP8 models: packed E4M3 [Mp][round512(H)] (padding zero)
  uint8_t* a8_dn = nullptr;    // packed E4M3 [Mp][round512(F)] (padding zero)
  float* sa_gu = nullptr;      // [Mp] row scales
  float* sa_dn = nullptr;
  uint32_t* rowmax_dn = nullptr;  // [Mp] SwiGLU row maxima (float bits)
};

// Bytes of a VerifyWs for n_branches x L rows of this model (regions aligned
// to 256 bytes), and the carving of such a buffer at base.
size_t verify_ws_bytes(const lopa_model* m, int32_t n_branches, int32_t L);
VerifyWs verify_ws_carve(const lopa_model* m, int32_t n_branches, int32_t L, char* base);
// Zero the padding columns of the carved operands (the GEMMs read them against
// zero weights; they must hold zeros, not stale values): a fill kernel, no
// memset node, so the call can sit in a captured graph.
int verify_ws_clear_padding(const lopa_model* m, int32_t n_branches, int32_t L, const VerifyWs& ws,
                            hipStream_t s);
// lopa_verify_forward with the working buffers ws instead of the KV handle's.
int verify_with_ws(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                   const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                   int32_t* pred, void* stream, const VerifyWs& ws);
// The argument checks of lopa_verify_forward (host only; 0 or a LOPA_E* code
// with the message set).
int verify_check(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                 const int32_t* branch_tokens, int32_t n_branches, int32_t L, float* conf,
                 int32_t* pred);
// The device the model's weights live on.
int model_device(const lopa_model* m);
// Record an error message for lopa_last_error and return code.
int lopa_fail(int code, const char* fmt, ...);

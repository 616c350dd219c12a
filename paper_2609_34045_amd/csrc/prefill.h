// Internal interface of the chunked-prefill path (matrix cores).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace kf {

struct PrefillArgs {
  int H, nq, nkv, hd, F;
  float eps;
  int T;          // tokens in the chunk
  int pos0;       // position of the first token
  int user;       // the user's row of the KV cache
  KvPages kv;
  const float* rope_cos;  // [max_ctx][hd/2]
  const float* rope_sin;
  int* err_flag;  // sticky error bits (kErrF16Range for an fp16 activation, key or value out of range)
  hipStream_t stream;
};

struct PrefillLayer {
  const uint16_t *wqkv, *wo, *wg, *wu, *wd, *g_attn, *g_mlp;
  const uint16_t *g_qn, *g_kn;  // per-head q / k norm gains (qk_norm blocks), else NULL
  uint16_t* kc;  // K cache of this layer (fp16 bits), pages as in KvPages
  uint16_t* vc;
  void* out;     // hidden output after this layer (last layer only), else NULL
  int out_bf16;
};

// Device workspace, grown on demand to the largest chunk seen.
struct PrefillWorkspace {
  int cap_T = 0;
  char* mem = nullptr;
  float* x = nullptr;      // [T][H] residual stream
  uint16_t* xn = nullptr;  // [T][H] normalised, fp16
  float* part = nullptr;   // split-K partial sums [slices][T][N] of the last split projection
  int pending = 0;         // slices of the down projection in `part` not yet added to x
  uint16_t* q = nullptr;   // [T][nq][hd] rotated queries, fp16
  uint16_t* o = nullptr;   // [T][nq hd] attention output, fp16
  uint16_t* act = nullptr; // [T][F] SwiGLU output, fp16
};

// Grows ws (hipMalloc) to hold a chunk of a.T tokens.
hipError_t prefill_reserve(PrefillWorkspace& ws, const PrefillArgs& a);
void prefill_free(PrefillWorkspace& ws);
// Device bytes a chunk of a.T tokens needs, and the workspace laid out from `base`
// (at least that many bytes, 256-byte aligned; ws does not own it).
int64_t prefill_ws_bytes(const PrefillArgs& a);
void prefill_carve(PrefillWorkspace& ws, char* base, const PrefillArgs& a);
hipError_t prefill_layer(PrefillWorkspace& ws, const PrefillArgs& a, const PrefillLayer& l, const Tracer& tr);

// Matrix-core GEMM of the prefill projections (gemm.hip); K must be a multiple
// of 64 (the stage's hidden, ffn and query widths are), else hipErrorInvalidValue.
//   kGemmResidF32   C[M][N] += A W^T (unsplit; the residual stream)
//   kGemmSwiGLU     Cb[M][N/2] = silu(gate) * up in fp16, W the gate rows and W2 the up rows
//   kGemmPartialF32 K slice ks to C + ks*M*N (plain stores); the consumer adds the
//                   gemm_splitk(M, N, K) slices in order
enum GemmEpi : int { kGemmResidF32 = 1, kGemmSwiGLU = 2, kGemmPartialF32 = 3 };
int gemm_splitk(int M, int N, int K);
hipError_t launch_gemm(int epi, const uint16_t* A, const uint16_t* W, const uint16_t* W2, int M, int N, int K,
                       float* C, uint16_t* Cb, int* err_flag, hipStream_t s);

}  // namespace kf

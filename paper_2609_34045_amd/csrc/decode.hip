// Decode-path kernels for gfx950 (CDNA4): one token per user, batch 1..4.
//
// At this batch size a stage reads each weight once per step and does a
// handful of FLOPs per weight byte, so every matrix product here is an
// HBM-bound GEMV (Section V-A of the paper prices a stage by exactly these
// bytes).  The kernels therefore stream the weights (fp16, converted from the model's
// bf16 when the stage is created) with 16-byte non-temporal
// loads, keep the (tiny) activations in L1/L2, and fuse everything elementwise
// into the GEMV that produces or consumes it:
//   * RMSNorm is folded into the consuming GEMV: the same loop that multiplies
//     a weight chunk by the input chunk also accumulates sum(x^2), so the
//     normalisation costs no extra pass;  y = rsqrt(mean(x^2)+eps) * W (x * g).
//   * RoPE and the KV-cache append run in the QKV GEMV's epilogue: one
//     workgroup owns rows i and i + hd/2 of a head, the pair RoPE rotates.
//   * SwiGLU runs in the gate/up GEMV's epilogue; the residual add in the
//     O and down GEMVs' epilogues.
//   * The LM-head GEMV reduces (max, lowest index) per workgroup.
// Attention is split-KV over an fp16 cache, [user][kv_head][pos][hd]; each
// workgroup serves all query heads of one KV head, and a second small kernel
// merges the splits of each (row, KV head) (online-softmax rescaling).
#include <type_traits>

#include "kernels.h"

namespace kf {

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

#ifndef KF_GEMV_NT
#define KF_GEMV_NT 1
#endif
// Weights are read once per step: non-temporal loads keep them from displacing
// the small, reused activations in the caches.
__device__ __forceinline__ v4u ld_stream(const v4u* p) {
#if KF_GEMV_NT
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

__device__ __forceinline__ void bf16x8(const v4u w, float (&f)[8]) {
  f[0] = __uint_as_float(w.x << 16);
  f[1] = __uint_as_float(w.x & 0xffff0000u);
  f[2] = __uint_as_float(w.y << 16);
  f[3] = __uint_as_float(w.y & 0xffff0000u);
  f[4] = __uint_as_float(w.z << 16);
  f[5] = __uint_as_float(w.z & 0xffff0000u);
  f[6] = __uint_as_float(w.w << 16);
  f[7] = __uint_as_float(w.w & 0xffff0000u);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef float f2 __attribute__((ext_vector_type(2)));

// 8 fp16 (16 bytes) to fp32.
__device__ __forceinline__ void f16x8(const v4u w, float (&f)[8]) {
  const f8 v = __builtin_convertvector(__builtin_bit_cast(h8, w), f8);
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = v[i];
}

// As f16x8, for products against fp32 inputs at batch > 1: the empty asm keeps
// the conversions separate instructions, since folding each into every row's
// FMA (a mixed-precision FMA per product) is several times slower.
__device__ __forceinline__ void f16x8_apart(const v4u w, float (&f)[8]) {
  f16x8(w, f);
#pragma unroll
  for (int i = 0; i < 8; ++i) asm("" : "+v"(f[i]));
}

// fp32 to fp16 bits, round to nearest even.
__device__ __forceinline__ uint16_t f32_to_f16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

// Round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Reduce-scatter of N per-lane values over a 64-lane wave: after it, v[0] of
// lane l holds the wave total of value index (l >> (6 - log2 N)).  Each step
// trades half of the remaining values with the lane O apart, so N values cost
// N - 1 shuffles (plus the all-reduce of the last one over the lanes that
// share an index) instead of 6 N.
template <int N, int O>
struct Butterfly {
  static __device__ __forceinline__ void run(float* v, int lane) {
    const bool up = (lane & O) != 0;
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      const float keep = up ? v[i + N / 2] : v[i];
      const float send = up ? v[i] : v[i + N / 2];
      v[i] = keep + __shfl_xor(send, O);
    }
    Butterfly<N / 2, O / 2>::run(v, lane);
  }
};
template <int O>
struct Butterfly<1, O> {
  static __device__ __forceinline__ void run(float* v, int lane) {
    v[0] += __shfl_xor(v[0], O);
    Butterfly<1, O / 2>::run(v, lane);
  }
};
template <>
struct Butterfly<1, 0> {
  static __device__ __forceinline__ void run(float*, int) {}
};

constexpr int ilog2(int n) { return n <= 1 ? 0 : 1 + ilog2(n / 2); }

// Reductions over lane groups of 8 or 16 (one half or one whole 16-lane DPP row),
// result in every lane of the group.  DPP operands feed the ALU directly, without
// the LDS round trip of a lane shuffle: quad_perm swaps lanes 1 and 2 apart, then
// the half-row and row mirrors pair each lane with one in the other quad / half.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
constexpr int kDppRor8 = 0x128;  // row_ror:8, i.e. lane xor 8 within each row of 16

template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 8 || N == 16, "group of 8 or 16 lanes");
  v += dpp<kDppXor1>(v);
  v += dpp<kDppXor2>(v);
  v += dpp<kDppHalfMirror>(v);
  if (N == 16) v += dpp<kDppMirror>(v);
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// ------------------------------------------------------------------ GEMV
// Workgroup of 256 threads owns R output rows of every batch row; its threads
// stride over K in 16-byte chunks (thread t takes chunks t, t+256, ...), so
// each wave's loads of a row are 1 KB contiguous.
// U chunks of all R rows are in flight per thread before any is consumed: a
// larger U shortens the serial chain of memory round trips per workgroup
// (what bounds the small matrices), a smaller U saves registers (occupancy,
// what bounds the large ones).
// Weight row of local row r (0..R-1) of workgroup wg, and whether it is a
// real output row.  QKV workgroups take R/2 rotation pairs (i, i + hd/2) of
// one head, so RoPE is applied in the epilogue; SwiGLU workgroups take R/2
// gate rows and the R/2 up rows of the same outputs.
template <int R, int EPI>
__device__ __forceinline__ const uint16_t* gemv_row(const GemvParams& p, int wg, int r, bool& ok) {
  ok = true;
  if (EPI == kEpiQKV) {
    const int wg_per_head = p.hd / R, head = wg / wg_per_head, i0 = (wg % wg_per_head) * (R / 2);
    const int row = head * p.hd + (r < R / 2 ? i0 + r : p.hd / 2 + i0 + r - R / 2);
    return p.w0 + (int64_t)row * p.K;
  } else if (EPI == kEpiSwiGLU) {
    // R / 2 outputs per workgroup; unless R / 2 divides 64 (and so every
    // supported ffn), the last workgroup has rows past the end
    const int row = wg * (R / 2) + (r < R / 2 ? r : r - R / 2);
    ok = 64 % (R / 2) == 0 || row < p.N;
    return (r < R / 2 ? p.w0 : p.w1) + (int64_t)(ok ? row : 0) * p.K;
  } else {
    const int row = wg * R + r;
    ok = row < p.N;
    return p.w0 + (int64_t)(ok ? row : 0) * p.K;
  }
}

// Values an epilogue thread needs from memory, requested when the kernel
// starts so that no memory round trip is left after the reduction: the RoPE
// cos/sin of its rotation pair (QKV) or the residual value it updates.
struct EpiPre {
  float a, b;
};

template <int B, int R, int EPI>
__device__ __forceinline__ EpiPre gemv_epi_prefetch(const GemvParams& p, int wg, int tid) {
  EpiPre e{0.f, 0.f};
  if (EPI == kEpiQKV) {
    if (tid < (R / 2) * B) {
      const int wg_per_head = p.hd / R, head = wg / wg_per_head, i0 = (wg % wg_per_head) * (R / 2);
      const int r = tid / B, b = tid % B, half = p.hd / 2;
      if (head < p.nq + p.nkv) {
        e.a = p.rope_cos[(int64_t)p.pos[b] * half + i0 + r];
        e.b = p.rope_sin[(int64_t)p.pos[b] * half + i0 + r];
      }
    }
  } else if (EPI == kEpiResid) {
    if (tid < R * B) {
      const int r = tid / B, b = tid % B, row = wg * R + r;
      if (row < p.N) e.a = p.x[(int64_t)b * p.N + row];
    }
  }
  return e;
}

constexpr int kNoRow = 0x7fffffff;  // argmax partial of a workgroup whose logits were all NaN

// Epilogue of a workgroup's R x B dot products fin[r * B + b] (plus, when the
// launch normalises its input, fin[R * B + b] = sum of x_b^2 over K).  Runs
// on the T threads (index tid) that own the group, after fin is complete.
template <int B, int R, int EPI, bool NORM, int T>
__device__ __forceinline__ void gemv_epilogue(const GemvParams& p, int wg, const float* fin, int tid,
                                              const EpiPre& pre) {
  bool bad = false;  // an fp16 store out of range
  float rs[B];
#pragma unroll
  for (int b = 0; b < B; ++b) rs[b] = NORM ? 1.0f / sqrtf(fin[R * B + b] / (float)p.K + p.eps) : 1.0f;

  if (EPI == kEpiQKV) {
    if (tid < (R / 2) * B) {
      const int wg_per_head = p.hd / R, head = wg / wg_per_head, i0 = (wg % wg_per_head) * (R / 2);
      const int r = tid / B, b = tid % B;
      const float y1 = fin[r * B + b] * rs[b];
      const float y2 = fin[(r + R / 2) * B + b] * rs[b];
      const int hd = p.hd, half = hd / 2, i = i0 + r, pos = p.pos[b];
      if (p.kraw && head < p.nq + p.nkv) {  // raw q / k: their norm and RoPE follow in another kernel
        float* dst = head < p.nq ? p.q + (int64_t)b * p.nq * hd + head * hd
                                 : p.kraw + ((int64_t)b * p.nkv + head - p.nq) * hd;
        dst[i] = y1;
        dst[i + half] = y2;
      } else if (head < p.nq + p.nkv) {
        const float c = pre.a, s = pre.b;
        const float z1 = y1 * c - y2 * s, z2 = y2 * c + y1 * s;
        if (head < p.nq) {
          float* q = p.q + (int64_t)b * p.nq * hd + head * hd;
          q[i] = z1;
          q[i + half] = z2;
        } else {
          uint16_t* k = p.kc + kv_offset(p.kv, p.users[b], head - p.nq, pos, hd);
          k[i] = f16_checked(z1, bad);
          k[i + half] = f16_checked(z2, bad);
        }
      } else {
        uint16_t* v = p.vc + kv_offset(p.kv, p.users[b], head - p.nq - p.nkv, pos, hd);
        v[i] = f16_checked(y1, bad);
        v[i + half] = f16_checked(y2, bad);
      }
    }
  } else if (EPI == kEpiResid) {
    static_assert(EPI != kEpiResid || R * B <= T, "one residual row per thread");
    if (tid < R * B) {
      const int t = tid, r = t / B, b = t % B, row = wg * R + r;
      if (row < p.N) {
        const int64_t at = (int64_t)b * p.N + row;
        const float v = pre.a + fin[t];
        p.x[at] = v;
        if (p.out2) {
          if (p.out2_type == kOut2F32) reinterpret_cast<float*>(p.out2)[at] = v;
          else reinterpret_cast<uint16_t*>(p.out2)[at] = p.out2_type == kOut2BF16 ? f32_to_bf16(v) : f16_checked(v, bad);
        }
      }
    }
  } else if (EPI == kEpiSwiGLU) {
    if (tid < (R / 2) * B && (64 % (R / 2) == 0 || wg * (R / 2) + tid / B < p.N)) {
      const int r = tid / B, b = tid % B;
      const float gt = fin[r * B + b] * rs[b];
      const float up = fin[(r + R / 2) * B + b] * rs[b];
      const float a = gt / (1.0f + expf(-gt)) * up;
      const int64_t at = (int64_t)b * p.N + wg * (R / 2) + r;
      if (p.act16) reinterpret_cast<uint16_t*>(p.act)[at] = f16_checked(a, bad);
      else p.act[at] = a;
    }
  } else {  // kEpiLMHead
    if (p.logits) {
      for (int t = tid; t < R * B; t += T) {
        const int r = t / B, b = t % B, row = wg * R + r;
        if (row < p.N) p.logits[(int64_t)b * p.N + row] = fin[t] * rs[b];
      }
    }
    if (tid < B) {
      // (max, lowest row) over the workgroup's rows; a NaN logit is skipped and
      // reported, and a workgroup of NaN rows leaves (-inf, kNoRow)
      const int b = tid;
      float best = -INFINITY;
      int bidx = kNoRow;
      bool nan = false;
      for (int r = 0; r < R; ++r) {
        const float v = fin[r * B + b] * rs[b];
        if (wg * R + r >= p.N) break;
        if (v != v) nan = true;
        else if (v > best || bidx == kNoRow) {  // strict: the lower row keeps a tie
          best = v;
          bidx = wg * R + r;
        }
      }
      p.part_val[(int64_t)b * p.n_wg + wg] = best;
      p.part_idx[(int64_t)b * p.n_wg + wg] = bidx;
      raise_err(p.err_flag, nan, kErrNaNLogit);
    }
  }
  raise_err(p.err_flag, bad, kErrF16Range);
}

// Vector-ALU GEMV: each thread multiplies its 16-byte weight chunks by the
// fp32 input rows, so a row's 8 products per chunk cost 8 FMAs per batch row.
// Input chunk c (8 values) of batch row b taken from the stage input: an fp32
// or bf16 hidden row, or the embedding row of a token (NaN for a token outside
// [0, vocab)).  The conversions are exact.
__device__ __forceinline__ void stage_input_chunk(const GemvParams& p, int b, int c, v4f& lo, v4f& hi) {
  const int K = p.K;
  if (p.tokens) {
    const int tok = p.tokens[b];
    if (tok < 0 || tok >= p.vocab) {
      const float qn = __uint_as_float(0x7fc00000u);
      lo = hi = v4f{qn, qn, qn, qn};
      return;
    }
    float f[8];
    bf16x8(*reinterpret_cast<const v4u*>(p.embed + (int64_t)tok * K + c * 8), f);
    lo = v4f{f[0], f[1], f[2], f[3]};
    hi = v4f{f[4], f[5], f[6], f[7]};
  } else if (p.src_bf16) {
    float f[8];
    bf16x8(*reinterpret_cast<const v4u*>(reinterpret_cast<const uint16_t*>(p.src) + (int64_t)b * K + c * 8), f);
    lo = v4f{f[0], f[1], f[2], f[3]};
    hi = v4f{f[4], f[5], f[6], f[7]};
  } else {
    const v4f* q = reinterpret_cast<const v4f*>(reinterpret_cast<const float*>(p.src) + (int64_t)b * K + c * 8);
    lo = q[0];
    hi = q[1];
  }
}

#ifndef KF_GEMV_MIN_WAVES
#define KF_GEMV_MIN_WAVES 4
#endif
// The weight bytes in flight per CU scale with resident waves; at batch 3-4 the
// input rows and partial sums put the kernel just past 128 VGPRs (3 waves per
// SIMD), so the register budget is held to 4 waves there.  Smaller batches are
// left to the compiler (a cap costs the batch-1 gate/up kernel a wave).
// With NORM and GAIN false the norm's gain has been folded into the weight
// matrix's columns at stage init (W diag(g), rounded once to fp16): the input
// rows meet the weights as they are, and only the sum of squares is taken
// (from batch 2 by packed dot products of the fp16 inputs with themselves).
template <int B, int R, int U, int EPI, bool NORM, bool SRC = false, bool IN16 = false, bool GAIN = true>
__global__ __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(B >= 3 ? KF_GEMV_MIN_WAVES : 1)))
void gemv_kernel(const GemvParams p) {
  constexpr int T = 256;
  constexpr int NV = R * B + (NORM ? B : 0);
  constexpr int NVP = NV <= 8 ? 8 : NV <= 16 ? 16 : NV <= 32 ? 32 : 64;
  static_assert(NV <= 64, "too many partial sums per workgroup");
  constexpr int LPI = 64 / NVP;  // lanes sharing one reduced value

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wg = blockIdx.x;
  const int K = p.K, nch = K >> 3;

  const v4u* wrow[R];
  bool rok[R];
#pragma unroll
  for (int r = 0; r < R; ++r) wrow[r] = reinterpret_cast<const v4u*>(gemv_row<R, EPI>(p, wg, r, rok[r]));
  const EpiPre pre = gemv_epi_prefetch<B, R, EPI>(p, wg, tid);
  if (SRC && wg == 0 && p.tokens && tid < B && (p.tokens[tid] < 0 || p.tokens[tid] >= p.vocab))
    atomicOr(p.err_flag, kErrToken);

  float acc[NVP];
#pragma unroll
  for (int i = 0; i < NVP; ++i) acc[i] = 0.f;

  // Load order within a chunk step (loads return in order): input rows (and
  // gain) first lets the norm and the first rows' FMAs start while the later
  // weight rows arrive; measured faster at batch > 1 and for QKV, while the
  // batch-1 gate/up and down launches are faster with the weights first.
  constexpr bool kInputFirst = B > 1 || EPI == kEpiQKV;
  // fp16 inputs (batch 2-4) meet the fp16 weights in packed dot products: two
  // products per instruction, summed in fp32.
  constexpr bool kDot = IN16 && !SRC;
  // From batch 2 the first layer's QKV launch rounds the stage input to fp16, as
  // the residual copy every later layer's QKV launch reads was rounded, and takes
  // the same packed products: a layer's result then does not depend on whether
  // it starts the stage (a stage split anywhere composes to the same output).
  constexpr bool kDotSrc = SRC && B > 1 && EPI == kEpiQKV;
  bool bad_in = false;  // a stage input value beyond the fp16 range (kDotSrc)
  for (int c0 = tid; c0 < nch; c0 += T * U) {
    v4f xl[U][B], xh[U][B];
    v4u xr[U][B];
    v4u gv[U];
    v4u wv[U][R];
    auto load_input = [&]() {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = (c0 + u * T < nch ? c0 + u * T : c0);  // past the end: re-read chunk c0, unused
#pragma unroll
        for (int b = 0; b < B; ++b) {
          if (SRC) {
            stage_input_chunk(p, b, c, xl[u][b], xh[u][b]);
          } else if (kDot) {
            xr[u][b] = *reinterpret_cast<const v4u*>(reinterpret_cast<const uint16_t*>(p.in) + (int64_t)b * K + c * 8);
          } else if (IN16) {  // 8 fp16 inputs (16 bytes), converted exactly
            float f[8];
            f16x8(*reinterpret_cast<const v4u*>(reinterpret_cast<const uint16_t*>(p.in) + (int64_t)b * K + c * 8), f);
            xl[u][b] = v4f{f[0], f[1], f[2], f[3]};
            xh[u][b] = v4f{f[4], f[5], f[6], f[7]};
          } else {
            const v4f* src = reinterpret_cast<const v4f*>(p.in + (int64_t)b * K + c * 8);
            xl[u][b] = src[0];
            xh[u][b] = src[1];
          }
        }
        if (NORM && GAIN) gv[u] = *reinterpret_cast<const v4u*>(p.gain + c * 8);
      }
    };
    if (kInputFirst) load_input();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * T;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (c < nch && rok[r]) wv[u][r] = ld_stream(wrow[r] + c);
        else wv[u][r] = v4u{0u, 0u, 0u, 0u};
      }
    }
    if (!kInputFirst) load_input();
    // every load of the chunk is issued before any arithmetic on it (left to
    // itself the scheduler may sink each weight load to its first use, which
    // leaves one 16-byte load per thread in flight)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * T;
      if (c < nch) {
        if (SRC && wg == 0 && p.x_init) {  // the residual stream starts as the stage input
#pragma unroll
          for (int b = 0; b < B; ++b) {
            reinterpret_cast<v4f*>(p.x_init + (int64_t)b * K + c * 8)[0] = xl[u][b];
            reinterpret_cast<v4f*>(p.x_init + (int64_t)b * K + c * 8)[1] = xh[u][b];
          }
        }
        if constexpr (kDot || kDotSrc) {
          // input pairs in fp16; with the norm, x * gain rounded to fp16 (sum(x^2) in fp32)
          h2 xp[B][4];
          float gf[8];
          if (NORM && GAIN) bf16x8(gv[u], gf);
          if constexpr (kDotSrc) {
#pragma unroll
            for (int b = 0; b < B; ++b) {
              const v4f lo = xl[u][b], hi = xh[u][b];
              const float xs[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
              uint16_t x16[8];
#pragma unroll
              for (int i = 0; i < 8; ++i) x16[i] = f16_checked(xs[i], bad_in);
              xr[u][b] = v4u{x16[0] | ((uint32_t)x16[1] << 16), x16[2] | ((uint32_t)x16[3] << 16),
                             x16[4] | ((uint32_t)x16[5] << 16), x16[6] | ((uint32_t)x16[7] << 16)};
            }
          }
#pragma unroll
          for (int b = 0; b < B; ++b) {
            if (NORM && GAIN) {
              float f[8];
              f16x8_apart(xr[u][b], f);
#pragma unroll
              for (int i = 0; i < 8; ++i) acc[R * B + b] += f[i] * f[i];
#pragma unroll
              for (int j = 0; j < 4; ++j) xp[b][j] = __builtin_convertvector(f2{f[2 * j] * gf[2 * j], f[2 * j + 1] * gf[2 * j + 1]}, h2);
            } else {
              const h8 x8 = __builtin_bit_cast(h8, xr[u][b]);
              xp[b][0] = __builtin_shufflevector(x8, x8, 0, 1);
              xp[b][1] = __builtin_shufflevector(x8, x8, 2, 3);
              xp[b][2] = __builtin_shufflevector(x8, x8, 4, 5);
              xp[b][3] = __builtin_shufflevector(x8, x8, 6, 7);
              if (NORM) {  // the gain is in the weights: the squares of the fp16 inputs, summed in fp32
                float q = acc[R * B + b];
#pragma unroll
                for (int j = 0; j < 4; ++j) q = __builtin_amdgcn_fdot2(xp[b][j], xp[b][j], q, false);
                acc[R * B + b] = q;
              }
            }
          }
#pragma unroll
          for (int r = 0; r < R; ++r) {
            const h8 w8 = __builtin_bit_cast(h8, wv[u][r]);
            const h2 w0 = __builtin_shufflevector(w8, w8, 0, 1), w1 = __builtin_shufflevector(w8, w8, 2, 3),
                     w2 = __builtin_shufflevector(w8, w8, 4, 5), w3 = __builtin_shufflevector(w8, w8, 6, 7);
#pragma unroll
            for (int b = 0; b < B; ++b) {
              float a = acc[r * B + b];
              a = __builtin_amdgcn_fdot2(w0, xp[b][0], a, false);
              a = __builtin_amdgcn_fdot2(w1, xp[b][1], a, false);
              a = __builtin_amdgcn_fdot2(w2, xp[b][2], a, false);
              acc[r * B + b] = __builtin_amdgcn_fdot2(w3, xp[b][3], a, false);
            }
          }
          continue;
        }
        float xf[B][8];
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const v4f lo = xl[u][b], hi = xh[u][b];
          xf[b][0] = lo.x; xf[b][1] = lo.y; xf[b][2] = lo.z; xf[b][3] = lo.w;
          xf[b][4] = hi.x; xf[b][5] = hi.y; xf[b][6] = hi.z; xf[b][7] = hi.w;
        }
        if (NORM) {
          float gf[8];
          if (GAIN) bf16x8(gv[u], gf);
#pragma unroll
          for (int b = 0; b < B; ++b) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              acc[R * B + b] += xf[b][i] * xf[b][i];
              if (GAIN) xf[b][i] *= gf[i];
            }
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float wf[8];
          if (B > 1) f16x8_apart(wv[u][r], wf);
          else f16x8(wv[u][r], wf);
#pragma unroll
          for (int b = 0; b < B; ++b) {
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[r * B + b] += wf[i] * xf[b][i];
          }
        }
      }
    }
  }

  if (kDotSrc) raise_err(p.err_flag, bad_in && wg == 0, kErrF16Range);
  Butterfly<NVP, 32>::run(acc, lane);
  __shared__ float red[4][NVP];
  __shared__ float fin[NVP];
  if ((lane & (LPI - 1)) == 0) red[wave][lane / LPI] = acc[0];
  __syncthreads();
  if (tid < NVP) fin[tid] = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
  __syncthreads();
  gemv_epilogue<B, R, EPI, NORM, T>(p, wg, fin, tid, pre);
}

// ------------------------------------------------------------------ attention
// Split-KV decode attention with the products on 16x16 MFMAs.  A workgroup
// (split s, KV head g, row b) covers keys [s*split, min((s+1)*split, len_b))
// for all G query heads of the group, so each K/V byte is read once per KV
// head, and writes the split's partial (max, sum, unnormalised acc).  Per block of 16 keys: S^T = K Q^T (16 keys x 16 query slots: the G
// heads of the group, zero-padded) and O^T += V^T P^T.  Wave w of the NW-wave
// workgroup takes the split's blocks w, w + NW, ...; each block's K and V rows
// come into a two-stage LDS ring of the wave's own by direct global->LDS loads,
// so the next block is in flight while one is computed, and the waves need no
// barrier until the final merge of their states.  K fragments are plain
// 16-byte LDS reads (lane l: key l % 16, one 16-byte chunk); V^T fragments are
// transpose reads (lane l: 4 keys of one d).  The score tile's lane layout
// (lane l: keys 4 (l / 16) .. + 3 of head l % 16) is exactly the P^T operand
// of the P V MFMA, so the softmax moves no data besides the maximum and the sum
// over the four 16-lane groups that share a head: a few vector instructions
// per key, where a vector-ALU kernel spent ~30 on dot products, 16-lane
// reductions and packed P V.  For blocks with per-head q/k norms it also
// normalises and rotates the queries and the new key.  Splits may start
// anywhere on a 16-key boundary; from batch 2 the host sizes them for about one
// workgroup per CU.  Measured against a deeper ring with K fragments read
// straight from memory (16 rows x 64 bytes per load: slower), eight-wave
// workgroups one per CU, and a split score chain with early V^T reads (both
// no faster).
namespace {
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void* dk_lds_ptr;

// Wait until at most N of this wave's vector memory operations are outstanding
// (direct loads count until their LDS write is done).
template <int N>
__device__ __forceinline__ void dk_wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(N | (0x7 << 4) | (0xF << 8));
}

// Slot of 16-byte chunk c of key row r in a block tile.  A K fragment read
// takes one chunk of 16 consecutive rows per 16 lanes, a V transpose read two
// neighbouring chunks of 8 consecutive rows per 32 lanes; f(r) puts both on
// distinct 16-byte bank groups of the 64-bank LDS (HD 64: two rows per line).
template <int HD>
__device__ __forceinline__ int dk_slot(int r, int c) {
  return HD == 128 ? c ^ (((r & 7) << 1) | ((r >> 3) & 1)) : c ^ ((((r >> 1) & 3) << 1) | ((r >> 3) & 1));
}

// max / sum of x over lanes l and l ^ 16 (permlane16_swap with x in both
// operands leaves x[l] and x[l ^ 16] in the two results), and over l and l ^ 32.
__device__ __forceinline__ float dk_max16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float dk_max32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float dk_sum16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float dk_sum32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint32_t dk_pack(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
}

// V^T fragments of one block: transpose reads at LDS byte addresses base + off[t].
// They are issued as inline assembly, followed by an explicit wait for their
// results: the compiler would otherwise wait for every direct load in flight
// (including the next block's) before the first transpose read.  The wait takes
// the results as operands, so no use of them can be scheduled above it.
template <int NT>
__device__ __forceinline__ void dk_read_vt(uint32_t base, const int (&off)[NT], v2u (&vf)[NT]) {
#pragma unroll
  for (int t = 0; t < NT; ++t)
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(vf[t]) : "v"(base + off[t]) : "memory");
  if constexpr (NT == 8)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(vf[0]), "+v"(vf[1]), "+v"(vf[2]), "+v"(vf[3]), "+v"(vf[4]), "+v"(vf[5]), "+v"(vf[6]),
                   "+v"(vf[7])::"memory");
  else
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(vf[0]), "+v"(vf[1]), "+v"(vf[2]), "+v"(vf[3])::"memory");
}
}  // namespace

#ifndef KF_ATTN_LAZY
#define KF_ATTN_LAZY 8.0f
#endif

template <int HD, int NW>
__global__ __launch_bounds__(64 * NW, NW >= 8 ? 1 : 2) void attn_decode_mfma_kernel(const AttnParams p) {
  constexpr int KB = 16;             // keys per block
  constexpr int ROWB = HD * 2;       // bytes per key row
  constexpr int CPR = ROWB / 16;     // 16-byte chunks per row
  constexpr int TILEB = KB * ROWB;   // K (or V) of one block
  constexpr int STAGEB = 2 * TILEB;  // K tile, then V tile
  constexpr int WAVEB = 2 * STAGEB;  // two stages per wave
  constexpr int LPT = TILEB / 1024;  // direct loads (1 KB per wave) per tile
  constexpr int RPL = 1024 / ROWB;   // key rows per direct load
  constexpr int NS = HD / 32;        // S MFMA steps (32 d each)
  constexpr int NT = HD / 16;        // O^T tiles (16 d each)
  constexpr float kLazy = KF_ATTN_LAZY;
  static_assert(HD == 64 || HD == 128, "head dim");
  static_assert(kKvPage % KB == 0 && kAttnMaxSplit / kKvPage <= 64, "blocks within pages");
  static_assert(HD * 16 * 4 + 32 * 4 <= WAVEB, "a wave's final state fits its stages");
  static_assert(NW * WAVEB <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NW * WAVEB];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = p.nq / p.nkv;  // query heads per KV head, at most 16
  const int hq0 = g * G;
  const int hn = lane & 15, q4 = lane >> 4;  // MFMA column (query slot) and 16-lane group

  // The query slots as fp16 B operands, scaled to log2 units: slot hn, d = 32 s + 8 q4 .. + 7
  // (requested first: the previous kernel has just written them).
  v4f qlo[NS], qhi[NS];
  {
    const bool hv = hn < G;
    const float* qr = p.q + (int64_t)b * p.nq * HD + (int64_t)(hq0 + (hv ? hn : 0)) * HD;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const v4f* src = reinterpret_cast<const v4f*>(qr + 32 * s + 8 * q4);
      qlo[s] = src[0];
      qhi[s] = src[1];
    }
  }
  asm volatile("" ::: "memory");  // the query loads go out before the exit test below
  const int len = p.len[b];
  const int s0 = split * p.split;
  const int nk = min(s0 + p.split, len) - s0;
  if (nk <= 0) {  // a trailing split of a shorter row: its partial is empty, (max, sum, acc) = (-inf, 0, 0)
    for (int e = tid; e < G * HD; e += 64 * NW) {
      const int h = e / HD, d = e % HD;
      const int64_t row = ((int64_t)b * p.nq + hq0 + h) * p.max_split + split;
      p.part_acc[row * HD + d] = 0.f;
      if (d == 0) {
        p.part_ml[row * 2] = -INFINITY;
        p.part_ml[row * 2 + 1] = 0.f;
      }
    }
    return;
  }
  const int nb = (nk + KB - 1) / KB;
  const int cw = nb > wave ? (nb - wave + NW - 1) / NW : 0;  // this wave's blocks: wave + NW i, i < cw
  const int u = p.users[b];
  uint8_t* region = smem + wave * WAVEB;

  // A paged cache's page ids for the split (at most kAttnMaxSplit / kKvPage + 1:
  // the split starts at key kp0 of its first page), lane i holding the split's
  // page i.  A block (16 keys, 16-aligned) lies in one page.
  const int kp0 = s0 % kKvPage, pg0 = s0 / kKvPage;
  int pid = 0;
  if (p.kv.table && lane * kKvPage < kp0 + nk) pid = p.kv.table[u * p.kv.ppu + pg0 + lane];
  auto block_off = [&](int blk) -> int64_t {  // element offset of the block's first key row
    const int k = kp0 + blk * KB, i = k / kKvPage;
    const int page = p.kv.table ? __builtin_amdgcn_readlane(pid, i) : u * p.kv.ppu + pg0 + i;
    return (int64_t)page * p.kv.page_stride + ((int64_t)g * kKvPage + k % kKvPage) * HD;
  };
  // Direct load j of a tile fills rows RPL j ..; lane l writes row RPL j + l / CPR,
  // slot l % CPR, so it fetches the chunk that belongs in that slot.  Rows past
  // the split's last key repeat that key (a written row of the same page): their
  // scores are masked, and their values stay finite.
  int drow[LPT], dchunk[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    drow[j] = RPL * j + lane / CPR;
    dchunk[j] = dk_slot<HD>(drow[j], lane % CPR) * 16;
  }
  auto issue = [&](int i) {  // this wave's block i into stage i % 2
    const int blk = NW * i + wave;
    const int64_t off = block_off(blk);
    const int last = nk - 1 - blk * KB;
    uint8_t* st = region + (i & 1) * STAGEB;
    const char* kb = reinterpret_cast<const char*>(p.kc + off);
    const char* vb = reinterpret_cast<const char*>(p.vc + off);
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const uint32_t byte = min(drow[j], last) * ROWB + dchunk[j];  // unsigned: a scalar base plus a 32-bit lane offset
      // (named operands: the host pass drops the kernel's launch stub when a
      // builtin's pointer argument is a compound expression)
      const char* ks = kb + byte;
      const char* vs = vb + byte;
      uint8_t* kd = st + 1024 * j;
      uint8_t* vd = st + TILEB + 1024 * j;
      __builtin_amdgcn_global_load_lds(ks, (dk_lds_ptr)kd, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vs, (dk_lds_ptr)vd, 16, 0, 0);
    }
  };
  if (cw > 0) issue(0);
  if (cw > 1) issue(1);

  // Blocks with per-head q/k norms: q comes raw from the QKV GEMV.  Each query
  // slot is RMS-normalised (gains gq; its squares summed over the four lanes
  // that hold it) and rotated at the row's new position: the RoPE partner of
  // d = 32 s + 8 q4 + j, d +- HD/2, is step s +- NS/2 of the same lane.
  const bool qkn = p.kraw != nullptr;
  const int npos = len - 1;  // row b's new position
  if (qkn) {
    float x[NS][8];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      x[s][0] = qlo[s].x; x[s][1] = qlo[s].y; x[s][2] = qlo[s].z; x[s][3] = qlo[s].w;
      x[s][4] = qhi[s].x; x[s][5] = qhi[s].y; x[s][6] = qhi[s].z; x[s][7] = qhi[s].w;
    }
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int j = 0; j < 8; ++j) ss += x[s][j] * x[s][j];
    const float rs = 1.0f / sqrtf(dk_sum32(dk_sum16(ss)) / (float)HD + p.eps);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      float gf[8];
      bf16x8(*reinterpret_cast<const v4u*>(p.gq + 32 * s + 8 * q4), gf);
#pragma unroll
      for (int j = 0; j < 8; ++j) x[s][j] *= rs * gf[j];
    }
#pragma unroll
    for (int s = 0; s < NS / 2; ++s) {
      const v4f* cp = reinterpret_cast<const v4f*>(p.rope_cos + (int64_t)npos * (HD / 2) + 32 * s + 8 * q4);
      const v4f* sp = reinterpret_cast<const v4f*>(p.rope_sin + (int64_t)npos * (HD / 2) + 32 * s + 8 * q4);
      const v4f c0 = cp[0], c1 = cp[1], n0 = sp[0], n1 = sp[1];
      const float c[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
      const float sn[8] = {n0.x, n0.y, n0.z, n0.w, n1.x, n1.y, n1.z, n1.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float a = x[s][j], bb = x[s + NS / 2][j];
        x[s][j] = a * c[j] - bb * sn[j];
        x[s + NS / 2][j] = bb * c[j] + a * sn[j];
      }
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qlo[s] = v4f{x[s][0], x[s][1], x[s][2], x[s][3]};
      qhi[s] = v4f{x[s][4], x[s][5], x[s][6], x[s][7]};
    }
  }
  // The new key of such a block: the wave whose block holds position npos
  // normalises (gains gk) and rotates it from its raw projection, lane c < CPR
  // taking 16-byte chunk c (partner chunk c +- CPR/2); it stores it to the cache
  // for later steps and writes it over that row of its LDS tile once the
  // block's direct loads have landed (the cache row they read was stale).
  const int rel_new = npos - s0;
  const bool own_new = qkn && rel_new >= 0 && rel_new < nk && (rel_new / KB) % NW == wave;
  const int i_new = own_new ? (rel_new / KB) / NW : -1;
  v4u knew = {0u, 0u, 0u, 0u};
  if (own_new) {
    const int c = lane % CPR, d0 = 8 * c;
    const v4f* src = reinterpret_cast<const v4f*>(p.kraw + ((int64_t)b * p.nkv + g) * HD + d0);
    const v4f lo = src[0], hi = src[1];
    float x[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    float gf[8];
    bf16x8(*reinterpret_cast<const v4u*>(p.gk + d0), gf);
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) ss += x[j] * x[j];
    const float rs = 1.0f / sqrtf(group_sum<CPR>(ss) / (float)HD + p.eps);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] *= rs * gf[j];
    const int i0 = d0 % (HD / 2);
    const float sgn = d0 < HD / 2 ? -1.f : 1.f;
    float y[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) y[j] = CPR == 16 ? dpp<kDppRor8>(x[j]) : __shfl_xor(x[j], CPR / 2);
    bool bad = false;
    uint16_t k16[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float cs = p.rope_cos[(int64_t)npos * (HD / 2) + i0 + j], sn = p.rope_sin[(int64_t)npos * (HD / 2) + i0 + j];
      k16[j] = f16_checked(x[j] * cs + sgn * y[j] * sn, bad);
    }
    knew = v4u{k16[0] | ((uint32_t)k16[1] << 16), k16[2] | ((uint32_t)k16[3] << 16),
               k16[4] | ((uint32_t)k16[5] << 16), k16[6] | ((uint32_t)k16[7] << 16)};
    if (lane < CPR) {
      *reinterpret_cast<v4u*>(p.kc + kv_offset(p.kv, u, g, npos, HD) + d0) = knew;
      raise_err(p.err_flag, bad, kErrF16Range);
    }
  }

  h8 qf[NS];
  {
    const float sc = hn < G ? p.scale_log2 : 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[s] = h8{(_Float16)(qlo[s].x * sc), (_Float16)(qlo[s].y * sc), (_Float16)(qlo[s].z * sc),
                 (_Float16)(qlo[s].w * sc), (_Float16)(qhi[s].x * sc), (_Float16)(qhi[s].y * sc),
                 (_Float16)(qhi[s].z * sc), (_Float16)(qhi[s].w * sc)};
  }
  // Fragment offsets within a stage.  K, step s: row hn, chunk 4 s + q4.  V^T,
  // tile t: key row 4 q4 + (lane / 4) % 4, d = 16 t + 4 (lane % 4) .. + 3.
  int koff[NS], voff[NT];
#pragma unroll
  for (int s = 0; s < NS; ++s) koff[s] = hn * ROWB + dk_slot<HD>(hn, 4 * s + q4) * 16;
  {
    const int key = 4 * q4 + ((lane >> 2) & 3), j = lane & 3;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int dd = 16 * t + 4 * j;
      voff[t] = key * ROWB + dk_slot<HD>(key, dd >> 3) * 16 + (dd & 7) * 2;
    }
  }
  const uint32_t region_lds = (uint32_t)(uintptr_t)(dk_lds_ptr)region;

  v4f o[NT];  // O^T tile t: lane holds d = 16 t + 4 q4 + r of query slot hn
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = v4f{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};

  for (int i = 0; i < cw; ++i) {
    if (i + 1 < cw) dk_wait_vm<2 * LPT>();  // block i has landed; block i + 1 may be in flight
    else dk_wait_vm<0>();
    asm volatile("" ::: "memory");  // no LDS read of the block moves above the wait
    const uint8_t* st = region + (i & 1) * STAGEB;
    if (i == i_new && lane < CPR)  // the new key over its stale row (this wave's reads follow in order)
      *reinterpret_cast<v4u*>(region + (i & 1) * STAGEB + (rel_new % KB) * ROWB + dk_slot<HD>(rel_new % KB, lane) * 16) = knew;
    v4f sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const v4u kf = *reinterpret_cast<const v4u*>(st + koff[s]);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, kf), qf[s], sc, 0, 0, 0);
    }
    const int k0 = (NW * i + wave) * KB + 4 * q4;  // this lane's first key, relative to the split
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (k0 + r >= nk) sc[r] = -INFINITY;
    // Online softmax.  The reference maximum moves only when the block's
    // maximum exceeds it by more than kLazy (log2 units), so probabilities stay
    // below 2^kLazy (fp16 holds them as exactly as values below 1) and the
    // rescale of O is skipped in nearly every block.  A block always holds a
    // valid key, so its maximum is finite.
    float mb = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    mb = dk_max32(dk_max16(mb));
    const float m_new = mb > m_run + kLazy ? mb : m_run;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 while m_run is -inf
    const uint32_t w0 = dk_pack(__builtin_amdgcn_exp2f(sc[0] - m_new), __builtin_amdgcn_exp2f(sc[1] - m_new));
    const uint32_t w1 = dk_pack(__builtin_amdgcn_exp2f(sc[2] - m_new), __builtin_amdgcn_exp2f(sc[3] - m_new));
    // the sum is taken over the fp16 probabilities that the P V product uses
    const float ls = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w1), ones,
                                            __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w0), ones, 0.f, false), false);
    l_run = l_run * alpha + ls;
    m_run = m_new;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
      for (int t = 0; t < NT; ++t) o[t] *= alpha;
    }
    v2u vf[NT];
    dk_read_vt<NT>(region_lds + (uint32_t)((i & 1) * STAGEB + TILEB), voff, vf);
    const h4 pf = __builtin_bit_cast(h4, v2u{w0, w1});
#pragma unroll
    for (int t = 0; t < NT; ++t)
      o[t] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(h4, vf[t]), pf, o[t], 0, 0, 0);
    if (i + 2 < cw) issue(i + 2);  // into the stage just read
  }
  l_run = dk_sum32(dk_sum16(l_run));  // over the four key groups of the head

  // The waves' states (O^T [d][slot], then max and sum per slot) meet in LDS
  // and are merged into the split's partial (max, sum, unnormalised acc).
  float* sw = reinterpret_cast<float*>(region);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) sw[(16 * t + 4 * q4 + r) * 16 + hn] = o[t][r];
  if (q4 == 0) {
    sw[HD * 16 + hn] = m_run;
    sw[HD * 16 + 16 + hn] = l_run;
  }
  __syncthreads();
  for (int e = tid; e < G * HD; e += 64 * NW) {
    const int h = e / HD, d = e % HD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, reinterpret_cast<const float*>(smem + w * WAVEB)[HD * 16 + h]);
    float v = 0.f, l = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float* s = reinterpret_cast<const float*>(smem + w * WAVEB);
        const float f = exp2f(s[HD * 16 + h] - M);  // 0 for a wave without keys (its max is -inf)
        v += f * s[d * 16 + h];
        l += f * s[HD * 16 + 16 + h];
      }
    }
    const int64_t row = ((int64_t)b * p.nq + hq0 + h) * p.max_split + split;
    p.part_acc[row * HD + d] = v;
    if (d == 0) {
      p.part_ml[row * 2] = M;
      p.part_ml[row * 2 + 1] = l;
    }
  }
}

// Merge of the split-KV partials of one (head h, row b): weights 2^(m_s - M)
// over the splits that saw keys (M their largest max), the weighted partial
// vectors summed and divided by the weighted partial sums.  The split weights are
// computed by all threads at once and kept in LDS; then each wave sums every
// fourth split's vector (independent loads) and the four sums are combined.  The
// result goes out for the output projection's GEMV: in fp16 (o16, batch > 1) or
// fp32 (o32, the batch-1 launch sequence that adds the heads in a fixed order).
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(const AttnParams a, uint16_t* __restrict__ o16,
                                                         float* __restrict__ o32) {
  constexpr int DPL = HD / 64;
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ns = a.n_split;
  const int64_t r0 = ((int64_t)b * a.nq + h) * a.max_split;
  const float* ml = a.part_ml + r0 * 2;
  const float* acc = a.part_acc + r0 * HD + lane * DPL;
  __shared__ float wsm[kAttnMaxSplitCount];
  __shared__ float red[4][HD];
  __shared__ float sM[4], sL[4];

  // Wave w's first PRE splits (w, w + 4, ...) are requested with the (max, sum)
  // pairs, so the weighted sum needs no second memory round trip; splits past
  // ns re-read split ns - 1 (in bounds, finite) and get weight 0 below.
  constexpr int PRE = 8;
  float pre[PRE][DPL];
#pragma unroll
  for (int k = 0; k < PRE; ++k) {
    const int sp = min(wave + 4 * k, ns - 1);
#pragma unroll
    for (int i = 0; i < DPL; ++i) pre[k][i] = acc[(int64_t)sp * HD + i];
  }

  float M = -INFINITY;
  for (int s = tid; s < ns; s += 256)
    if (ml[2 * s + 1] > 0.f) M = fmaxf(M, ml[2 * s]);
  M = wave_max(M);
  if (lane == 0) sM[wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(sM[0], sM[1]), fmaxf(sM[2], sM[3]));
  float L = 0.f;
  for (int s = tid; s < ns; s += 256) {
    const float l = ml[2 * s + 1];
    const float w = l > 0.f ? __builtin_amdgcn_exp2f(ml[2 * s] - M) : 0.f;  // no keys: weight 0
    wsm[s] = w;
    L += w * l;
  }
  L = wave_sum(L);
  if (lane == 0) sL[wave] = L;
  __syncthreads();

  float o[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) o[i] = 0.f;
#pragma unroll
  for (int k = 0; k < PRE; ++k) {
    const int sp = wave + 4 * k;
    const float w = sp < ns ? wsm[sp] : 0.f;
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] += w * pre[k][i];
  }
#pragma unroll 8
  for (int s = wave + 4 * PRE; s < ns; s += 4) {
    const float w = wsm[s];
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] += w * acc[(int64_t)s * HD + i];
  }
#pragma unroll
  for (int i = 0; i < DPL; ++i) red[wave][lane * DPL + i] = o[i];
  __syncthreads();
  if (wave == 0) {
    const float inv = 1.0f / ((sL[0] + sL[1]) + (sL[2] + sL[3]));  // every row has at least one key
    const int64_t at = ((int64_t)b * a.nq + h) * HD + lane * DPL;
    bool bad = false;
#pragma unroll
    for (int i = 0; i < DPL; ++i) {
      const int d = lane * DPL + i;
      const float v = ((red[0][d] + red[1][d]) + (red[2][d] + red[3][d])) * inv;
      if (o16) o16[at + i] = f16_checked(v, bad);
      else o32[at + i] = v;
    }
    raise_err(a.err_flag, bad, kErrF16Range);
  }
}

// Output projection fused with the merge of the split-KV partials.  Workgroup
// (row block rb, query head h) merges head h's partials of every batch row
// into o_h in LDS (wave b takes row b: weights 2^(m_s - M) per split, sum of
// the weighted partial vectors, divided by the weighted sum of the partial
// denominators) and adds W_o[rows, h*hd:(h+1)*hd] o_h to the residual rows
// with fp32 atomics: the nq heads of a row arrive in any order.  A row's
// slice is read by 16 lanes x 16 bytes, so every load reads whole rows.  The
// merging waves request their partials (L2- or cache-resident, written by the
// attention kernel just before) ahead of the weights: loads return in order,
// so the merge runs while the weights are still on their way from HBM.
template <int B, int HD>
__global__ __launch_bounds__(256) void oproj_heads_kernel(const AttnParams a, const uint16_t* __restrict__ w,
                                                          float* __restrict__ x, int N) {
  constexpr int LPR = HD / 8;            // lanes per row
  constexpr int RPI = 64 / LPR;          // rows per wave-wide load
  constexpr int RPW = kOprojRows / 4;    // rows per wave
  constexpr int IT = RPW / RPI;          // loads per lane
  static_assert(IT >= 1 && IT <= LPR && (IT & (IT - 1)) == 0, "a power of two of reduced rows per row group");
  constexpr int LPV = LPR / IT;          // lanes holding each reduced row
  constexpr int DPL = HD / 64, PRE = 32;
  const int rb = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.nq * HD, ns = a.n_split;
  const int row0 = rb * kOprojRows + wave * RPW + lane / LPR;
  const int c8 = (lane % LPR) * 8;
  __shared__ float so[B][HD];
  __shared__ float wsplit[B][kAttnMaxSplitCount];

  // merging waves: the first PRE splits' partial vectors and the first 64 splits' (max, sum)
  const int b = wave < B ? wave : 0;
  const int64_t r0 = ((int64_t)b * a.nq + h) * a.max_split;
  const float* acc = a.part_acc + r0 * HD + lane * DPL;
  const float* ml = a.part_ml + r0 * 2;
  float pre[PRE][DPL];
  float m0 = -INFINITY, l0 = 0.f;
  if (wave < B) {
    // splits past ns re-read split ns-1 (in bounds) and get weight 0 below
#pragma unroll
    for (int sp = 0; sp < PRE; ++sp) {
      const float* src = acc + (int64_t)(sp < ns ? sp : ns - 1) * HD;
      if (DPL == 2) {
        const float2 v = *reinterpret_cast<const float2*>(src);
        pre[sp][0] = v.x;
        pre[sp][DPL - 1] = v.y;
      } else {
        pre[sp][0] = src[0];
      }
    }
    const float2 v = *reinterpret_cast<const float2*>(ml + 2 * (lane < ns ? lane : ns - 1));
    m0 = v.x;
    l0 = v.y;  // lanes past ns are masked after the weight loads are issued
  }

  v4u wv[IT];
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const int row = min(row0 + i * RPI, N - 1);  // rows past N load row N-1; their sums are dropped
    wv[i] = ld_stream(reinterpret_cast<const v4u*>(w + (int64_t)row * K + h * HD + c8));
  }

  if (wave < B) {
    if (lane >= ns) l0 = 0.f;
    // splits without keys carry (max, sum) = (-inf, 0) and get weight 0
    float M = l0 > 0.f ? m0 : -INFINITY;
    for (int s = lane + 64; s < ns; s += 64)
      if (ml[2 * s + 1] > 0.f) M = fmaxf(M, ml[2 * s]);
    M = wave_max(M);
    float L = 0.f;
    {
      const float ws = l0 > 0.f ? exp2f(m0 - M) : 0.f;
      if (lane < ns) wsplit[b][lane] = ws;
      L = ws * l0;
    }
    for (int s = lane + 64; s < ns; s += 64) {
      const float l = ml[2 * s + 1];
      const float ws = l > 0.f ? exp2f(ml[2 * s] - M) : 0.f;
      wsplit[b][s] = ws;
      L += ws * l;
    }
    L = wave_sum(L);
    float o[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = 0.f;
#pragma unroll
    for (int sp = 0; sp < PRE; ++sp) {
      const float ws = sp < ns ? wsplit[b][sp] : 0.f;
#pragma unroll
      for (int i = 0; i < DPL; ++i) o[i] += ws * pre[sp][i];
    }
#pragma unroll 8
    for (int sp = PRE; sp < ns; ++sp) {
      const float ws = wsplit[b][sp];
#pragma unroll
      for (int i = 0; i < DPL; ++i) o[i] += ws * acc[(int64_t)sp * HD + i];
    }
    const float inv = 1.0f / L;
#pragma unroll
    for (int i = 0; i < DPL; ++i) so[b][lane * DPL + i] = o[i] * inv;
  }
  __syncthreads();

  float ov[B][8];
#pragma unroll
  for (int bb = 0; bb < B; ++bb)
#pragma unroll
    for (int e = 0; e < 8; ++e) ov[bb][e] = so[bb][c8 + e];
  float sum[B][IT];
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    float wf[8];
    f16x8(wv[i], wf);
#pragma unroll
    for (int bb = 0; bb < B; ++bb) {
      float t = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) t += wf[e] * ov[bb][e];
      sum[bb][i] = t;
    }
  }
  // lanes LPV j .. LPV j + LPV - 1 of a row group end with the group total of load j: row row0 + j * RPI
  const int j = (lane % LPR) / LPV, row = row0 + j * RPI;
#pragma unroll
  for (int bb = 0; bb < B; ++bb) {
    Butterfly<IT, LPR / 2>::run(sum[bb], lane);
    if (row < N && lane % LPV == 0) atomicAdd(x + (int64_t)bb * N + row, sum[bb][0]);
  }
}

// ------------------------------------------------------------------ small kernels
// One thread per 4 elements of the [rows][H] input (H is a multiple of 64).
__global__ void prep_hidden_kernel(const void* __restrict__ in, int in_bf16, const int32_t* __restrict__ tokens,
                                   const uint16_t* __restrict__ embed, int vocab, float* __restrict__ x, int rows, int H,
                                   int* err_flag) {
  const int64_t i4 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;  // index of a group of 4 elements
  const int64_t n4 = (int64_t)rows * H / 4;
  if (i4 >= n4) return;
  const int row = (int)(i4 * 4 / H), k = (int)(i4 * 4 % H);
  v4f v;
  if (tokens) {
    const int tok = tokens[row];
    if (tok < 0 || tok >= vocab) {
      if (k == 0) atomicOr(err_flag, kErrToken);
      const float qn = __uint_as_float(0x7fc00000u);
      v = v4f{qn, qn, qn, qn};
    } else {
      const uint2 e = *reinterpret_cast<const uint2*>(embed + (int64_t)tok * H + k);
      v = v4f{__uint_as_float(e.x << 16), __uint_as_float(e.x & 0xffff0000u), __uint_as_float(e.y << 16),
              __uint_as_float(e.y & 0xffff0000u)};
    }
  } else if (in_bf16) {
    const uint2 e = reinterpret_cast<const uint2*>(in)[i4];
    v = v4f{__uint_as_float(e.x << 16), __uint_as_float(e.x & 0xffff0000u), __uint_as_float(e.y << 16),
            __uint_as_float(e.y & 0xffff0000u)};
  } else {
    v = reinterpret_cast<const v4f*>(in)[i4];
  }
  reinterpret_cast<v4f*>(x)[i4] = v;
}

// Second level of the greedy argmax: the per-workgroup (max, lowest row) pairs
// of one batch row reduced by one 1024-thread workgroup.  Each thread requests
// U = 16 pairs before comparing any, so up to 16,384 pairs per row (every LM
// head grid up to V = 131,072 at 8 rows per workgroup) take one memory round trip.
__device__ __forceinline__ void argmax_take(float v, int ix, float& best, int& bidx) {
  if (v > best || (v == best && ix < bidx)) {
    best = v;
    bidx = ix;
  }
}

__global__ __launch_bounds__(1024) void argmax_final_kernel(const float* part_val, const int* part_idx, int n_wg,
                                                            int32_t* token, float* max_logit) {
  constexpr int T = 1024, U = 16;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* pv = part_val + (int64_t)b * n_wg;
  const int* pi = part_idx + (int64_t)b * n_wg;
  float best = -INFINITY;
  int bidx = kNoRow;
  for (int i0 = tid; i0 < n_wg; i0 += T * U) {
    float v[U];
    int ix[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * T;
      v[u] = i < n_wg ? pv[i] : -INFINITY;
      ix[u] = i < n_wg ? pi[i] : kNoRow;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) argmax_take(v[u], ix[u], best, bidx);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) argmax_take(__shfl_xor(best, o), __shfl_xor(bidx, o), best, bidx);
  __shared__ float sv[T / 64];
  __shared__ int si[T / 64];
  if (lane == 0) {
    sv[wave] = best;
    si[wave] = bidx;
  }
  __syncthreads();
  if (wave == 0) {
    best = lane < T / 64 ? sv[lane] : -INFINITY;
    bidx = lane < T / 64 ? si[lane] : kNoRow;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) argmax_take(__shfl_xor(best, o), __shfl_xor(bidx, o), best, bidx);
    if (lane == 0) {
      token[b] = bidx == kNoRow ? -1 : bidx;  // -1: every logit of the row was NaN (kErrNaNLogit is raised)
      if (max_logit) max_logit[b] = bidx == kNoRow ? __builtin_nanf("") : best;
    }
  }
}

// In place: bf16 bits -> fp16 bits, round to nearest even.  Raises *bad when a
// finite value lies beyond the fp16 range (it would become infinite).
__global__ void weights_to_f16_kernel(uint16_t* w, int64_t n, int* bad) {
  int flag = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float v = bf16_to_f32(w[i]);
    const _Float16 h = (_Float16)v;
    flag |= __builtin_isinf((float)h) && !__builtin_isinf(v);
    w[i] = __builtin_bit_cast(uint16_t, h);
  }
  if (flag) atomicOr(bad, 1);
}

// Whether every fp16 rounding of w[r][k] g[k] (bf16 w [rows][K] and g [K]) is
// finite: flag set when one is not (its gain then stays out of the matrix).
__global__ void gain_fold_check_kernel(const uint16_t* w, int64_t n, int K, const uint16_t* g, int* flag) {
  int over = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float v = bf16_to_f32(w[i]) * bf16_to_f32(g[i % K]);  // exact in fp32 (8-bit significands)
    over |= __builtin_isinf((float)(_Float16)v) && !__builtin_isnan(v);
  }
  if (over) atomicOr(flag, 1);
}

// In place: bf16 w[r][k] -> fp16 bits of w[r][k] g[k], rounded to nearest even
// (the norm's gain folded into the matrix's columns).  Raises *bad when a
// product lies beyond the fp16 range, and, as for a matrix stored without its
// gain, when a finite weight itself does (whatever its gain).
__global__ void weights_to_f16_gain_kernel(uint16_t* w, int64_t n, int K, const uint16_t* g, int* bad) {
  int flag = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float x = bf16_to_f32(w[i]), v = x * bf16_to_f32(g[i % K]);
    const _Float16 h = (_Float16)v;
    flag |= __builtin_isinf((float)h) && !__builtin_isinf(v) && !__builtin_isnan(v);
    flag |= __builtin_isinf((float)(_Float16)x) && !__builtin_isinf(x);
    w[i] = __builtin_bit_cast(uint16_t, h);
  }
  if (flag) atomicOr(bad, 1);
}

__global__ void store_hidden_kernel(const float* x, void* out, int out_bf16, int64_t n) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (out_bf16) reinterpret_cast<uint16_t*>(out)[i] = f32_to_bf16(x[i]);
  else reinterpret_cast<float*>(out)[i] = x[i];
}

// src [n][nkv][hd] -> the cache at positions pos0 .. pos0 + n - 1 of one user, stored as fp16.
__global__ void kv_write_kernel(uint16_t* dk, uint16_t* dv, const KvPages kp, int user, int pos0, const void* sk,
                                const void* sv, int src_type, int n, int nkv, int hd) {
  const int64_t total = (int64_t)n * nkv * hd;
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % hd);
  const int g = (int)((i / hd) % nkv);
  const int t = (int)(i / ((int64_t)hd * nkv));
  const int64_t at = kv_offset(kp, user, g, pos0 + t, hd) + d;
  if (src_type == 2) {
    dk[at] = reinterpret_cast<const uint16_t*>(sk)[i];
    dv[at] = reinterpret_cast<const uint16_t*>(sv)[i];
  } else if (src_type == 1) {
    dk[at] = f32_to_f16(bf16_to_f32(reinterpret_cast<const uint16_t*>(sk)[i]));
    dv[at] = f32_to_f16(bf16_to_f32(reinterpret_cast<const uint16_t*>(sv)[i]));
  } else {
    dk[at] = f32_to_f16(reinterpret_cast<const float*>(sk)[i]);
    dv[at] = f32_to_f16(reinterpret_cast<const float*>(sv)[i]);
  }
}

__global__ void kv_read_kernel(const uint16_t* sk, const uint16_t* sv, const KvPages kp, int user, int pos0, float* dk,
                               float* dv, int n, int nkv, int hd) {
  const int64_t total = (int64_t)n * nkv * hd;
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int d = (int)(i % hd);
  const int g = (int)((i / hd) % nkv);
  const int t = (int)(i / ((int64_t)hd * nkv));
  const int64_t at = kv_offset(kp, user, g, pos0 + t, hd) + d;
  dk[i] = (float)__builtin_bit_cast(_Float16, sk[at]);
  dv[i] = (float)__builtin_bit_cast(_Float16, sv[at]);
}

__global__ void kv_table_update_kernel(int* table, const KvTableUpdate u) {
  const int i = threadIdx.x;
  if (i < u.n) table[u.idx[i]] = u.val[i];
}

// ------------------------------------------------------------------ launchers
// A launch that folds RMSNorm into its product: with the gain (p.gain) applied
// to the input rows, or, with p.gain NULL, already folded into the weights.
template <int B, int R, int U, int EPI, bool SRC, bool IN16>
static void gemv_norm_launch(const GemvParams& p, int grid, hipStream_t s) {
  if (p.gain) hipLaunchKernelGGL((gemv_kernel<B, R, U, EPI, true, SRC, IN16, true>), dim3(grid), dim3(256), 0, s, p);
  else hipLaunchKernelGGL((gemv_kernel<B, R, U, EPI, true, SRC, IN16, false>), dim3(grid), dim3(256), 0, s, p);
}

template <int B, int R, int U>
static hipError_t gemv_dispatch_epi(int epi, bool norm, const GemvParams& p, int grid, hipStream_t s) {
  if (epi == kEpiQKV && norm && B > 1 && p.in16)
    gemv_norm_launch<B, R, U, kEpiQKV, false, (B > 1)>(p, grid, s);
  else if (epi == kEpiQKV && norm && !p.in16)
    gemv_norm_launch<B, R, U, kEpiQKV, false, false>(p, grid, s);
  else if (epi == kEpiResid && !norm && B > 1 && p.in16)
    hipLaunchKernelGGL((gemv_kernel<B, R, U, kEpiResid, false, false, (B > 1)>), dim3(grid), dim3(256), 0, s, p);
  else if (epi == kEpiResid && !norm && !p.in16)
    hipLaunchKernelGGL((gemv_kernel<B, R, U, kEpiResid, false>), dim3(grid), dim3(256), 0, s, p);
  else if (epi == kEpiSwiGLU && norm && B > 1 && p.in16)
    gemv_norm_launch<B, R, U, kEpiSwiGLU, false, (B > 1)>(p, grid, s);
  else if (epi == kEpiSwiGLU && norm && !p.in16)
    gemv_norm_launch<B, R, U, kEpiSwiGLU, false, false>(p, grid, s);
  else if (epi == kEpiLMHead && norm && B > 1 && p.in16)
    gemv_norm_launch<B, R, U, kEpiLMHead, false, (B > 1)>(p, grid, s);
  else if (epi == kEpiLMHead && norm && !p.in16)
    gemv_norm_launch<B, R, U, kEpiLMHead, false, false>(p, grid, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int B, int R, int U>
static hipError_t gemv_dispatch_src(int epi, bool norm, const GemvParams& p, int grid, hipStream_t s) {
  if (epi == kEpiQKV && norm)
    gemv_norm_launch<B, R, U, kEpiQKV, true, false>(p, grid, s);
  else if (epi == kEpiLMHead && norm)
    gemv_norm_launch<B, R, U, kEpiLMHead, true, false>(p, grid, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int R, int U, bool SRC>
static hipError_t gemv_dispatch_b(int epi, bool norm, const GemvParams& p, int grid, hipStream_t s) {
  switch (p.batch) {
    case 1: return SRC ? gemv_dispatch_src<1, R, U>(epi, norm, p, grid, s) : gemv_dispatch_epi<1, R, U>(epi, norm, p, grid, s);
    case 2: return SRC ? gemv_dispatch_src<2, R, U>(epi, norm, p, grid, s) : gemv_dispatch_epi<2, R, U>(epi, norm, p, grid, s);
    case 3: return SRC ? gemv_dispatch_src<3, R, U>(epi, norm, p, grid, s) : gemv_dispatch_epi<3, R, U>(epi, norm, p, grid, s);
    case 4: return SRC ? gemv_dispatch_src<4, R, U>(epi, norm, p, grid, s) : gemv_dispatch_epi<4, R, U>(epi, norm, p, grid, s);
    default: return hipErrorInvalidValue;
  }
}

int gemv_grid(int epi, int R, const GemvParams& p) {
  switch (epi) {
    case kEpiQKV: return (p.nq + 2 * p.nkv) * (p.hd / R);
    case kEpiSwiGLU: return (p.N + R / 2 - 1) / (R / 2);
    default: return (p.N + R - 1) / R;
  }
}

hipError_t launch_gemv_src(int epi, int R, int U, bool norm, const GemvParams& p, hipStream_t s) {
  if ((p.src == nullptr) == (p.tokens == nullptr)) return hipErrorInvalidValue;
  const int grid = gemv_grid(epi, R, p);
  if (R == 8 && U == 1) return gemv_dispatch_b<8, 1, true>(epi, norm, p, grid, s);
  return hipErrorInvalidValue;
}

// Residual GEMV in workgroups of 4 or 10 rows (fp16 inputs from batch 2, as at 8 rows).
template <int B, int R>
static hipError_t resid_launch(const GemvParams& p, int grid, hipStream_t s) {
  if (B > 1 && p.in16)
    hipLaunchKernelGGL((gemv_kernel<B, R, 1, kEpiResid, false, false, (B > 1)>), dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((gemv_kernel<B, R, 1, kEpiResid, false>), dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}
template <int R>
static hipError_t resid_dispatch_b(const GemvParams& p, int grid, hipStream_t s) {
  switch (p.batch) {
    case 1: return resid_launch<1, R>(p, grid, s);
    case 2: return resid_launch<2, R>(p, grid, s);
    case 3: return resid_launch<3, R>(p, grid, s);
    case 4: return resid_launch<4, R>(p, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemv(int epi, int R, int U, bool norm, const GemvParams& p, hipStream_t s) {
  const int grid = gemv_grid(epi, R, p);
  if (R == 8 && U == 1) return gemv_dispatch_b<8, 1, false>(epi, norm, p, grid, s);
  if (R == 4 && U == 1 && epi == kEpiResid && !norm) return resid_dispatch_b<4>(p, grid, s);
  // The LM head on fp16 input rows (batch 2-4) in workgroups of 12 rows.
  if (R == 12 && U == 1 && epi == kEpiLMHead && norm && p.in16) {
    switch (p.batch) {
      case 2: gemv_norm_launch<2, 12, 1, kEpiLMHead, false, true>(p, grid, s); break;
      case 3: gemv_norm_launch<3, 12, 1, kEpiLMHead, false, true>(p, grid, s); break;
      case 4: gemv_norm_launch<4, 12, 1, kEpiLMHead, false, true>(p, grid, s); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (R == 10 && U == 1 && epi == kEpiResid && !norm) return resid_dispatch_b<10>(p, grid, s);
  // Batch-1 QKV in workgroups of 4 rows (2 rotation pairs): twice the workgroups
  // of the 8-row launch, which measured 0.1 us faster per layer at the 8B shape.
  if (R == 4 && U == 1 && epi == kEpiQKV && p.batch == 1 && norm && !p.in16) {
    gemv_norm_launch<1, 4, 1, kEpiQKV, false, false>(p, grid, s);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attn_decode(const AttnParams& p, int batch, hipStream_t s) {
  if (p.nq % p.nkv || p.nq / p.nkv > 16) return hipErrorInvalidValue;  // query slots of one MFMA column block
  const dim3 grid(p.n_split, p.nkv, batch);
  if (p.hd == 128)
    hipLaunchKernelGGL((attn_decode_mfma_kernel<128, kAttnMfmaWaves>), grid, dim3(64 * kAttnMfmaWaves), 0, s, p);
  else if (p.hd == 64)
    hipLaunchKernelGGL((attn_decode_mfma_kernel<64, kAttnMfmaWaves>), grid, dim3(64 * kAttnMfmaWaves), 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int HD>
static hipError_t oproj_dispatch(const AttnParams& a, const uint16_t* w, float* x, int N, int batch, hipStream_t s) {
  const dim3 grid((N + kOprojRows - 1) / kOprojRows, a.nq);
  switch (batch) {
    case 1: hipLaunchKernelGGL((oproj_heads_kernel<1, HD>), grid, dim3(256), 0, s, a, w, x, N); break;
    case 2: hipLaunchKernelGGL((oproj_heads_kernel<2, HD>), grid, dim3(256), 0, s, a, w, x, N); break;
    case 3: hipLaunchKernelGGL((oproj_heads_kernel<3, HD>), grid, dim3(256), 0, s, a, w, x, N); break;
    case 4: hipLaunchKernelGGL((oproj_heads_kernel<4, HD>), grid, dim3(256), 0, s, a, w, x, N); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnParams& a, uint16_t* o16, float* o32, int batch, hipStream_t s) {
  if (batch < 1 || batch > kMaxBatch || (o16 == nullptr) == (o32 == nullptr)) return hipErrorInvalidValue;
  const dim3 grid(a.nq, batch);
  if (a.hd == 128) hipLaunchKernelGGL(attn_merge_kernel<128>, grid, dim3(256), 0, s, a, o16, o32);
  else if (a.hd == 64) hipLaunchKernelGGL(attn_merge_kernel<64>, grid, dim3(256), 0, s, a, o16, o32);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_oproj_heads(const AttnParams& a, const uint16_t* w, float* x, int N, int batch, hipStream_t s) {
  if (a.hd == 128) return oproj_dispatch<128>(a, w, x, N, batch, s);
  if (a.hd == 64) return oproj_dispatch<64>(a, w, x, N, batch, s);
  return hipErrorInvalidValue;
}

hipError_t launch_prep_hidden(const void* in, int in_bf16, const int32_t* tokens, const uint16_t* embed, int vocab,
                              float* x, int rows, int H, int* err_flag, hipStream_t s) {
  const int64_t n4 = (int64_t)rows * H / 4;
  hipLaunchKernelGGL(prep_hidden_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, in, in_bf16, tokens,
                     embed, vocab, x, rows, H, err_flag);
  return hipGetLastError();
}

hipError_t launch_argmax_final(const float* part_val, const int* part_idx, int n_wg, int rows, int32_t* token,
                               float* max_logit, hipStream_t s) {
  hipLaunchKernelGGL(argmax_final_kernel, dim3(rows), dim3(1024), 0, s, part_val, part_idx, n_wg, token, max_logit);
  return hipGetLastError();
}

hipError_t launch_weights_to_f16(uint16_t* w, int64_t n, int* bad, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(weights_to_f16_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0, s, w, n, bad);
  return hipGetLastError();
}

hipError_t launch_gain_fold_check(const uint16_t* w, int64_t n, int K, const uint16_t* g, int* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(gain_fold_check_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0, s, w, n, K, g,
                     flag);
  return hipGetLastError();
}

hipError_t launch_weights_to_f16_gain(uint16_t* w, int64_t n, int K, const uint16_t* g, int* bad, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(weights_to_f16_gain_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0, s, w, n, K,
                     g, bad);
  return hipGetLastError();
}

hipError_t launch_store_hidden(const float* x, void* out, int out_bf16, int64_t n, hipStream_t s) {
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(store_hidden_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, out, out_bf16, n);
  return hipGetLastError();
}

hipError_t launch_kv_write(uint16_t* k, uint16_t* v, const KvPages& kp, int user, int pos0, const void* src_k,
                           const void* src_v, int src_type, int n, int nkv, int hd, hipStream_t s) {
  const int64_t total = (int64_t)n * nkv * hd;
  hipLaunchKernelGGL(kv_write_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, k, v, kp, user, pos0,
                     src_k, src_v, src_type, n, nkv, hd);
  return hipGetLastError();
}

hipError_t launch_kv_read(const uint16_t* k, const uint16_t* v, const KvPages& kp, int user, int pos0, float* dst_k,
                          float* dst_v, int n, int nkv, int hd, hipStream_t s) {
  const int64_t total = (int64_t)n * nkv * hd;
  hipLaunchKernelGGL(kv_read_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, k, v, kp, user, pos0,
                     dst_k, dst_v, n, nkv, hd);
  return hipGetLastError();
}

hipError_t launch_kv_table_update(int* table, const KvTableUpdate& u, hipStream_t s) {
  if (u.n < 1 || u.n > kKvTableBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kv_table_update_kernel, dim3(1), dim3(kKvTableBatch), 0, s, table, u);
  return hipGetLastError();
}

}  // namespace kf

// Chunked-prefill kernels for gfx950: a chunk of T tokens of one user.
//
// With T in the hundreds the projections are dense contractions,
// [T, K] x [N, K]^T, and run on the matrix cores (v_mfma_f32_32x32x16_f16:
// fp16 operands, fp32 accumulation).  Activations are kept in fp16 (8x the
// mantissa of bf16 at the same width), and the weights are held in fp16 since
// the stage was created.  A value stored in fp16 that reaches 65520 in
// magnitude raises the stage's range error bit.  Both operands are
// K-contiguous in HBM (activations row-major, weights [out, in]), so every
// MFMA operand fragment is one 16-byte run of a row.
// Attention is causal flash attention over the fp16 cache [0, pos0) plus the
// chunk, also on the matrix cores.
//
// Operand fragment layout of v_mfma_f32_32x32x16_f16 (lane l of 64):
//   A: row l%32, k = 8*(l/32) .. +7      B: column l%32, k = 8*(l/32) .. +7
//   D: element v (0..15) at row 8*(v/4) + 4*(l/32) + v%4, column l%32
#include <cmath>

#include "kernels.h"
#include <algorithm>
#include <type_traits>

#include "prefill.h"

namespace kf {

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float from_bf16(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Two fp32 to packed fp16 (round to nearest even).
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, h2));
}

// As pack_f16, noting in `bad` a value fp16 cannot hold (see f16_checked).
__device__ __forceinline__ uint32_t pack_f16_checked(float a, float b, bool& bad) {
  bad |= (__builtin_fabsf(a) >= 65520.0f) | (__builtin_fabsf(b) >= 65520.0f);
  return pack_f16(a, b);
}

__device__ __forceinline__ f32x16 mfma32(v4u a, v4u b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

// ------------------------------------------------------------------ row RMSNorm -> fp16
// Row RMSNorm of the residual stream to fp16 (gain g, or none when g is NULL:
// the gain is then folded into the next projection's weights).  With nsplit > 0 the row first
// takes the nsplit split-K slices of the projection that just ran (part, slice
// stride `stride`), added in slice order, and the sum is written back to x.
// Threads move 16 bytes at a time and request every slice before adding; the
// row loops are unrolled by 4, so the loads of four 16-byte steps are in flight
// together (70B-shaped rows: 24.6 -> 21.1 us per norm).
constexpr int kMaxSlices = 8;
#ifndef KF_PF_ATTN_SPLIT
#define KF_PF_ATTN_SPLIT 2  // key splits of the prefill attention when the chunk gives < 512 workgroups
#endif

__global__ __launch_bounds__(256) void rmsnorm_rows_f16_kernel(float* __restrict__ x, const float* __restrict__ part, int nsplit,
                                                                int64_t stride, const uint16_t* __restrict__ g, float eps,
                                                                uint16_t* __restrict__ out, int H, int* err_flag) {
  const int row = blockIdx.x, tid = threadIdx.x, H4 = H / 4;
  v4f* xr = reinterpret_cast<v4f*>(x + (int64_t)row * H);
  const v4f* pr = reinterpret_cast<const v4f*>(part + (int64_t)row * H);
  const int64_t st4 = stride / 4;
  float ss = 0.f;
#pragma unroll 4
  for (int k = tid; k < H4; k += 256) {
    v4f v = xr[k];
    if (nsplit > 0) {
      v4f sl[kMaxSlices];
#pragma unroll
      for (int i = 0; i < kMaxSlices; ++i)
        if (i < nsplit) sl[i] = pr[i * st4 + k];
#pragma unroll
      for (int i = 0; i < kMaxSlices; ++i)
        if (i < nsplit) v += sl[i];
      xr[k] = v;
    }
    ss += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  __shared__ float red[4];
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float rs = 1.0f / sqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)H + eps);
  uint2* o = reinterpret_cast<uint2*>(out + (int64_t)row * H);
  const uint2* g4 = reinterpret_cast<const uint2*>(g);
  bool bad = false;
#pragma unroll 4
  for (int k = tid; k < H4; k += 256) {
    const v4f v = xr[k] * rs;
    const uint2 gw = g4 ? g4[k] : uint2{0x3F803F80u, 0x3F803F80u};  // g NULL: folded into the next matrix (gain 1)
    o[k] = uint2{pack_f16_checked(v.x * __uint_as_float(gw.x << 16), v.y * __uint_as_float(gw.x & 0xffff0000u), bad),
                 pack_f16_checked(v.z * __uint_as_float(gw.y << 16), v.w * __uint_as_float(gw.y & 0xffff0000u), bad)};
  }
  raise_err(err_flag, bad, kErrF16Range);
}

// ------------------------------------------------------------------ RoPE + KV append
// QKV [T][(nq+2nkv) hd] fp32, the sum of nsplit split-K slices of `qkv` (slice
// stride `stride`) -> q [T][nq][hd] fp16 (rotated), K/V cache at pos0 + i (fp16).
// A thread takes 4 consecutive rotation pairs (j .. j+3, j+hd/2 .. j+hd/2+3).
// With gq / gk set (blocks with per-head q / k norms), each q and k head is
// RMS-normalised over its hd values first: the hd/8 consecutive threads that
// hold a head add their squares with lane shuffles.
__global__ __launch_bounds__(256) void rope_kv_kernel(const float* qkv, int nsplit, int64_t stride, uint16_t* q,
                                                      uint16_t* kc, uint16_t* vc, const KvPages kp, int user,
                                                      const float* cosT, const float* sinT, int nq, int nkv, int hd,
                                                      int pos0, const uint16_t* gq, const uint16_t* gk, float eps,
                                                      int* err_flag) {
  const int i = blockIdx.x, half = hd / 2, q4 = half / 4, pos = pos0 + i;
  const int nh = nq + 2 * nkv;
  const float* src = qkv + (int64_t)i * nh * hd;
  bool bad = false;
  for (int e = threadIdx.x; e < nh * q4; e += 256) {
    const int h = e / q4, j = (e % q4) * 4;
    v4f a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
    {
      v4f sa[kMaxSlices], sb[kMaxSlices];
#pragma unroll
      for (int sl = 0; sl < kMaxSlices; ++sl)
        if (sl < nsplit) {
          sa[sl] = *reinterpret_cast<const v4f*>(src + sl * stride + h * hd + j);
          sb[sl] = *reinterpret_cast<const v4f*>(src + sl * stride + h * hd + j + half);
        }
#pragma unroll
      for (int sl = 0; sl < kMaxSlices; ++sl)
        if (sl < nsplit) {
          a += sa[sl];
          b += sb[sl];
        }
    }
    uint16_t* dst;
    v4f z1, z2;
    if (gq && h < nq + nkv) {  // the q4 threads of a head are consecutive lanes of one wave
      float ss = a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
      for (int o = 1; o < q4; o <<= 1) ss += __shfl_xor(ss, o);
      const float rs = 1.0f / sqrtf(ss / (float)hd + eps);
      const uint16_t* g = h < nq ? gq : gk;
      const v4f ga = {from_bf16(g[j]), from_bf16(g[j + 1]), from_bf16(g[j + 2]), from_bf16(g[j + 3])};
      const v4f gb = {from_bf16(g[j + half]), from_bf16(g[j + half + 1]), from_bf16(g[j + half + 2]),
                      from_bf16(g[j + half + 3])};
      a = a * rs * ga;
      b = b * rs * gb;
    }
    if (h < nq + nkv) {
      const v4f c = *reinterpret_cast<const v4f*>(cosT + (int64_t)pos * half + j);
      const v4f s = *reinterpret_cast<const v4f*>(sinT + (int64_t)pos * half + j);
      z1 = a * c - b * s;
      z2 = b * c + a * s;
      dst = h < nq ? q + ((int64_t)i * nq + h) * hd : kc + kv_offset(kp, user, h - nq, pos, hd);
    } else {
      z1 = a;
      z2 = b;
      dst = vc + kv_offset(kp, user, h - nq - nkv, pos, hd);
    }
    *reinterpret_cast<uint2*>(dst + j) = uint2{pack_f16_checked(z1.x, z1.y, bad), pack_f16_checked(z1.z, z1.w, bad)};
    *reinterpret_cast<uint2*>(dst + j + half) =
        uint2{pack_f16_checked(z2.x, z2.y, bad), pack_f16_checked(z2.z, z2.w, bad)};
  }
  raise_err(err_flag, bad, kErrF16Range);
}

// ------------------------------------------------------------------ causal flash attention
// Workgroup = (128 queries, one query head); wave w owns queries 32w .. 32w+31.
// Per block of 64 keys each wave computes S^T = K Q^T (keys x queries) so that
// every lane holds one query's column; the online softmax is then per lane, and
// the lane's probabilities are already a B fragment of O^T += V^T P^T once the
// MFMA's k index is mapped to the keys the lane holds.
//
// K and V blocks go from the cache straight into LDS (global_load_lds) in their
// [key][d] layout, 16-byte chunks XOR-swizzled within a key row.  The V^T
// operand fragments are read with ds_read_b64_tr_b16: within each group of 16
// lanes, lane 4r + j reads 4 consecutive d of key row r and lane c receives
// element c of the group's four rows, i.e. d = d0 + c over 4 consecutive keys.
// The loop is software-pipelined: the S MFMAs of block j+1 are issued among
// the softmax of block j.  K and V have 2-stage rings of their own, each
// loaded one iteration ahead, right after the barrier that frees its stage.
//
// The keys may be split over gridDim.z workgroups (more workgroups in flight,
// two per CU): split z takes key blocks [z nblk / Z, (z+1) nblk / Z) and, when
// Z > 1, writes its unnormalised output and (max, sum) per query to part_acc /
// part_ml for attn_prefill_combine_kernel.
#ifndef KF_PF_ATTN_RING
#define KF_PF_ATTN_RING 4
#endif
constexpr int kRing = KF_PF_ATTN_RING;  // LDS fragment reads in flight ahead of the MFMAs
#ifndef KF_PF_ATTN_LAZY
#define KF_PF_ATTN_LAZY 8.0f
#endif
constexpr float kLazy = KF_PF_ATTN_LAZY;
constexpr int kAttnKB = 64;  // keys per block
typedef __attribute__((address_space(3))) void* lds_ptr;
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s* lds_v4s;

// Slot of 16-byte chunk c of key row r.  A K fragment read takes one chunk of
// 16 consecutive rows (HD 128) or of 8 same-parity rows among 16 (HD 64) per
// LDS cycle; a V transpose read takes 4 consecutive rows x 4 consecutive
// chunks.  f(r) puts both on distinct 16-byte bank groups of a 64-bank LDS.
template <int HD>
__device__ __forceinline__ int kv_slot(int r, int c) {
  return HD == 128 ? c ^ (((r & 3) << 2) | ((r >> 2) & 3)) : c ^ ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}

// max / sum of x over lanes l and l ^ 32: v_permlane32_swap with x in both
// operands leaves x[l] in one result and x[l ^ 32] in the other.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Wait until this wave's global loads (and the LDS writes of direct loads) are complete.
__device__ __forceinline__ void attn_wait_loads() { __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xF << 8)); }
// Workgroup barrier across which the compiler may not move memory operations.
__device__ __forceinline__ void attn_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_prefill_kernel(const uint16_t* q, const uint16_t* kc,
                                                           const uint16_t* vc, const KvPages kp, int user,
                                                           uint16_t* out, float* part_acc, float* part_ml, int T,
                                                           int nq, int nkv, int pos0, float scale_log2,
                                                           int* err_flag) {
  constexpr int KB = kAttnKB, NT = KB / 32;  // keys per block, 32-key tiles per block
  constexpr int NS = HD / 16, DB = HD / 32;  // 16-wide d slices of S, 32-row d blocks of O^T
  constexpr int CPR = HD / 8;                // 16-byte chunks per key row
  constexpr int ROWB = HD * 2;               // bytes per key row
  constexpr int TILEB = KB * ROWB;           // one block of K (or V): 16 KB (HD 128) or 8 KB
  constexpr int RPI = 64 / CPR;              // key rows per 1 KB direct load
  constexpr int LPW = TILEB / 1024 / 4;      // direct loads per wave per tile
  static_assert(HD == 64 || HD == 128, "head dim");
  static_assert(kKvPage % KB == 0, "key blocks within pages");
  // K stages 0 and 1, then V stages 0 and 1.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[4 * TILEB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Workgroups go to the 8 XCDs round-robin by linear id.  Numbering the work
  // XCD-major (logical id = xcd * n / 8 + slot) puts the workgroups of one KV
  // group on as few XCDs as possible, so that group's K and V stay in one L2.
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  {
    const int nx = gridDim.x, ny = gridDim.y, n = nx * ny * gridDim.z;
    const int lin = bx + nx * (by + ny * bz);
    if (n % 8 == 0) {
      const int l = (lin % 8) * (n / 8) + lin / 8;  // z slowest within a head, then query tile
      bz = l % gridDim.z;
      bx = (l / gridDim.z) % nx;
      by = l / (gridDim.z * nx);
    }
  }
  const int h = by, g = h / (nq / nkv);
  const int i0 = bx * 128;
  const int qi = i0 + wave * 32 + (lane & 31);  // this lane's query (chunk index)
  const int half_sel = lane >> 5;
  const bool qok = qi < T;
  const int qpos = pos0 + qi;
  const int last_q = min(i0 + 127, T - 1);
  const int nkeys = pos0 + last_q + 1;  // keys visible to the workgroup's last query
  const int nblk_all = (nkeys + KB - 1) / KB;
  const int Z = gridDim.z, z = bz;
  const int blk0 = (int)((int64_t)nblk_all * z / Z), blk1 = (int)((int64_t)nblk_all * (z + 1) / Z);
  // A block of KB keys lies in one cache page (KB divides kKvPage, blocks start at multiples of KB).
  // Page ids of a paged cache for blocks [pb, pb + 64) of the range, lane i
  // holding block pb + i's (a block is one page), loaded outside the loop's
  // issue points: a table load there would put a wait for every direct load
  // in flight in front of the next block's loads.
  static_assert(KB == kKvPage, "one page per key block");
  int pb = blk0, pid = 0;
  auto load_pids = [&]() {
    pid = (kp.table && pb + lane < kp.ppu) ? kp.table[user * kp.ppu + pb + lane] : 0;
  };
  load_pids();
  auto block_off = [&](int blk) -> int64_t {  // wave-uniform: the block's loads take a scalar base
    const int page = kp.table ? __builtin_amdgcn_readlane(pid, blk - pb) : user * kp.ppu + blk;
    return (int64_t)page * kp.page_stride + (int64_t)g * kKvPage * HD;
  };

  // Q^T fragments: lane holds query qi, d = 16 s + 8 half_sel .. +7.
  v4u qf[NS];
  {
    const uint16_t* qr = q + ((int64_t)(qok ? qi : 0) * nq + h) * HD;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      v4u v = *reinterpret_cast<const v4u*>(qr + 16 * s + 8 * half_sel);
      qf[s] = qok ? v : v4u{0u, 0u, 0u, 0u};
    }
  }

  f32x16 o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[d][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  auto kst = [&](int blk) { return smem + ((blk - blk0) & 1) * TILEB; };
  auto vst = [&](int blk) { return smem + (2 + ((blk - blk0) & 1)) * TILEB; };
  // Direct loads of block blk's K or V rows into a stage: load j of this wave
  // fills rows RPI (4 j + wave) ..; lane l writes row RPI (4 j + wave) + l / CPR,
  // slot l % CPR, so it fetches the chunk that belongs in that slot (byte
  // offset dma_off[j] within the block).  Keys at or past nkeys come after
  // every query of the workgroup, so the causal mask gives them weight 0; in
  // the block that holds nkeys - 1 they are loaded from that key instead, a
  // written row of the same page.
  // (unsigned lane offsets from the block's wave-uniform base: the loads take
  // the base in scalar registers and the offset as their 32-bit vector operand)
  int dma_row[LPW];
  uint32_t dma_chunk[LPW], dma_off[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    dma_row[j] = RPI * (4 * j + wave) + lane / CPR;
    dma_chunk[j] = kv_slot<HD>(dma_row[j], lane % CPR) * 16;
    dma_off[j] = dma_row[j] * ROWB + dma_chunk[j];
  }
  auto issue = [&](const uint16_t* cache, int blk, uint8_t* dst) {
    const int last = nkeys - 1 - blk * KB;
    const char* base = reinterpret_cast<const char*>(cache + block_off(blk));
    if (last >= KB - 1) {
#pragma unroll
      for (int j = 0; j < LPW; ++j) {
        const char* src = base + dma_off[j];
        uint8_t* d = dst + 1024 * (4 * j + wave);
        __builtin_amdgcn_global_load_lds(src, (lds_ptr)d, 16, 0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < LPW; ++j) {
        const char* src = base + (uint32_t)(min(dma_row[j], last) * ROWB + dma_chunk[j]);
        uint8_t* d = dst + 1024 * (4 * j + wave);
        __builtin_amdgcn_global_load_lds(src, (lds_ptr)d, 16, 0, 0);
      }
    }
  };

  // Lane byte offsets of the fragment reads within a stage.  The row swizzle
  // depends only on a row's low four bits, so the key tile and step add a
  // constant (an immediate of the read).
  //   K, slice s: row lane % 32 (+ 32 t), chunk 2 s + half_sel.
  //   V^T, d-block d and half e: key row 8 e + 4 (gq / 2) + r (+ 32 t + 16 sidx),
  //   d = 32 d + 16 (gq % 2) + 4 j, with lane = 16 gq + 4 r + j.
  int koff[NS], voff[DB][2];
  {
    const int rl = lane & 31;
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) koff[s2] = rl * ROWB + kv_slot<HD>(rl, 2 * s2 + half_sel) * 16;
    const int gq = lane >> 4, tr_r = (lane >> 2) & 3, tr_j = lane & 3;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = 8 * e + 4 * (gq >> 1) + tr_r, dd = 32 * d + 16 * (gq & 1) + 4 * tr_j;
        voff[d][e] = key * ROWB + kv_slot<HD>(key, dd >> 3) * 16 + (dd & 7) * 2;
      }
  }
  constexpr int NI_S = NT * NS;
  auto kread = [&](const uint8_t* ks, int i) {
    return *reinterpret_cast<const v4u*>(ks + (i / NS) * 32 * ROWB + koff[i % NS]);
  };

  // Causal mask of block blk's scores (only blocks that reach past the wave's
  // first query have masked keys).  Lane holds keys 32 t + 8 (v/4) + 4 half_sel
  // + v%4 of its query.
  auto mask = [&](int blk, f32x16 (&st)[NT]) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = blk * KB + 32 * t + 8 * (v >> 2) + 4 * half_sel + (v & 3);
        if (key > qpos) st[t][v] = -INFINITY;
      }
  };

  // Online softmax of a block's (masked, unscaled) scores st into the P^T
  // fragments pf; returns the factor O must be rescaled by.  The scale (> 0)
  // commutes with the maximum and is folded into the exponent's fma.  The row
  // sum is taken over the fp16 probabilities that the P V product uses.
  auto softmax = [&](f32x16 (&st)[NT], v4u (&pf)[NT][2]) {
    float mb = -INFINITY;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mb = fmaxf(mb, st[t][v]);
    mb = pair_max(mb);
    // The reference maximum moves only when the block's maximum exceeds it by
    // more than kLazy (log2 units): probabilities then stay below 2^kLazy,
    // which fp16 holds as exactly as values below 1, and the rescale of O
    // (and its multiplies) is skipped in nearly every block.  The result
    // O / l does not depend on the reference.
    const float m_blk = mb * scale_log2;
    const float m_new = m_blk > m_run + kLazy ? m_blk : m_run;
    // Until a visible key has been seen (possible in a later key split) the
    // maximum is -inf; 0 then stands in as reference so that every
    // probability, and the rescale of the empty state, is exactly 0.
    const float m_ref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);  // 0 while m_run = -inf
    float ls = 0.f;
    // P^T fragments of tile t: step 0 takes v = 0..7, step 1 takes v = 8..15 (the
    // MFMA's k index runs over the keys this lane holds, in that order).
    const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int v = 8 * sidx + 2 * e;
          w[e] = pack_f16(__builtin_amdgcn_exp2f(fmaf(st[t][v], scale_log2, -m_ref)),
                          __builtin_amdgcn_exp2f(fmaf(st[t][v + 1], scale_log2, -m_ref)));
          ls = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w[e]), ones, ls, false);
        }
        pf[t][sidx] = v4u{w[0], w[1], w[2], w[3]};
      }
    l_run = l_run * alpha + pair_sum(ls);
    m_run = m_new;
    return alpha;
  };

  // O^T += V^T P^T from block blk's V stage.  MFMA i: d-block i / NP, key step
  // (t, sidx) = i % NP, whose keys are 32 t + 16 sidx + 4 half_sel + {0..3} and
  // + 8 + {0..3} in the MFMA's k order: two transpose reads.
  auto pv_mfma = [&](const uint8_t* vs, const v4u (&pf)[NT][2]) {
    constexpr int NP = NT * 2, NI = DB * NP;
    auto vread = [&](int i) {
      const int d = i / NP, t = (i % NP) / 2, sidx = i % 2;
      // (named operands: the host pass drops the kernel's launch stub when a
      // builtin's pointer argument is a compound expression)
      const uint8_t* b = vs + (32 * t + 16 * sidx) * ROWB;
      const uint8_t* a0 = b + voff[d][0];
      const uint8_t* a1 = b + voff[d][1];
      const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)a0);
      const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)a1);
      const v2u l2 = __builtin_bit_cast(v2u, lo), h2v = __builtin_bit_cast(v2u, hi);
      return v4u{l2.x, l2.y, h2v.x, h2v.y};
    };
    v4u ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = vread(i);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      // the MFMA takes the slot before its refill is issued (no register copy)
      o[i / NP] = mfma32(ring[i % kRing], pf[(i % NP) / 2][i % 2], o[i / NP]);
      if (i + kRing < NI) ring[i % kRing] = vread(i + kRing);
    }
  };

  // S^T[key][query] of one block from its K stage.  The K fragments go through
  // a ring of kRing registers: the read for MFMA i + kRing is issued before
  // MFMA i, so LDS latency hides behind the MFMAs in flight.
  auto s_mfma = [&](const uint8_t* ks, f32x16 (&st)[NT]) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) st[t][v] = 0.f;
    v4u ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = kread(ks, i);
#pragma unroll
    for (int i = 0; i < NI_S; ++i) {
      st[i / NS] = mfma32(ring[i % kRing], qf[i % NS], st[i / NS]);
      if (i + kRing < NI_S) ring[i % kRing] = kread(ks, i + kRing);
    }
  };

  // The same S MFMAs with the softmax of the previous block's scores sc (as
  // softmax() computes it) spread over the MFMA slots, pinned in order, so
  // that the wave issues vector work while its MFMAs run: the block maximum
  // over the first quarter of the slots, the reference update in one slot,
  // the probabilities (exponent, fp16 pack, running sum) over the next half,
  // the row sum in one more.
  auto s_mfma_softmax = [&](const uint8_t* ks, f32x16 (&st)[NT], f32x16 (&sc)[NT], v4u (&pf)[NT][2]) {
    constexpr int NV = NT * 16;                 // scores per lane
    constexpr int MAXS = NI_S / 4, EXPS = NI_S / 2;
    constexpr int MPS = NV / MAXS, EPS = NV / EXPS;  // scores per slot in the max and exponent phases
    static_assert(MAXS + 1 + EXPS + 1 <= NI_S && NV % MAXS == 0 && NV % EXPS == 0 && EPS % 2 == 0, "phases");
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) st[t][v] = 0.f;
    float mb = -INFINITY, m_new = 0.f, m_ref = 0.f, alpha = 1.f, ls = 0.f;
    uint32_t w[NV / 2];
    const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};
    v4u ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = kread(ks, i);
#pragma unroll
    for (int i = 0; i < NI_S; ++i) {
      st[i / NS] = mfma32(ring[i % kRing], qf[i % NS], st[i / NS]);
      if (i + kRing < NI_S) ring[i % kRing] = kread(ks, i + kRing);
      if (i < MAXS) {
#pragma unroll
        for (int u = i * MPS; u < (i + 1) * MPS; ++u) mb = fmaxf(mb, sc[u / 16][u % 16]);
      } else if (i == MAXS) {
        mb = pair_max(mb);
        const float m_blk = mb * scale_log2;
        m_new = m_blk > m_run + kLazy ? m_blk : m_run;
        m_ref = m_new == -INFINITY ? 0.f : m_new;
        alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
      } else if (i <= MAXS + EXPS) {
        const int k = i - MAXS - 1;
#pragma unroll
        for (int u = k * EPS; u < (k + 1) * EPS; u += 2) {
          w[u / 2] = pack_f16(__builtin_amdgcn_exp2f(fmaf(sc[u / 16][u % 16], scale_log2, -m_ref)),
                              __builtin_amdgcn_exp2f(fmaf(sc[(u + 1) / 16][(u + 1) % 16], scale_log2, -m_ref)));
          ls = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w[u / 2]), ones, ls, false);
        }
      } else if (i == MAXS + EXPS + 1) {
        l_run = l_run * alpha + pair_sum(ls);
        m_run = m_new;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // word u/2 holds scores u, u+1 = (t, v) with v = 8 sidx + 2 e
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        const int b0 = (16 * t + 8 * sidx) / 2;
        pf[t][sidx] = v4u{w[b0], w[b0 + 1], w[b0 + 2], w[b0 + 3]};
      }
    return alpha;
  };

  // Iteration blk: on entry K(blk + 1) and V(blk) were loaded (by this wave)
  // an iteration ago, and S(blk) is in sc.  After the barrier every wave's
  // loads have landed and every wave is done with K(blk) (read for S(blk))
  // and V(blk - 1), so their stages take K(blk + 2) and V(blk + 1).  The
  // parity P of blk - blk0 is a compile-time constant, so every stage
  // address is a constant and the fragment reads take it as their immediate
  // offset (a stage chosen at run time cost a vector add per read).
  auto iteration = [&](auto parity, int blk, f32x16 (&sc)[NT], f32x16 (&sn)[NT]) {
    constexpr int P = decltype(parity)::value;
    uint8_t* const k_this = smem + P * TILEB;  // K(blk), then K(blk + 2)
    uint8_t* const k_next = smem + (1 - P) * TILEB;
    uint8_t* const v_this = smem + (2 + P) * TILEB;
    uint8_t* const v_next = smem + (3 - P) * TILEB;
    attn_wait_loads();
    attn_barrier();
    if (kp.table && blk + 2 >= pb + 64) {  // the window moves on (every 62 blocks)
      pb = blk + 1;
      load_pids();
    }
    if (blk + 2 < blk1) issue(kc, blk + 2, k_this);
    if (blk + 1 < blk1) issue(vc, blk + 1, v_next);
    if (blk * KB + KB - 1 > pos0 + i0 + wave * 32) mask(blk, sc);
    v4u pf[NT][2];
    float alpha;
    if (blk + 1 < blk1) alpha = s_mfma_softmax(k_next, sn, sc, pf);
    else alpha = softmax(sc, pf);
    if (__ballot(alpha != 1.0f)) {  // no lane's reference moved: nothing to rescale
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[d][v] *= alpha;
    }
    pv_mfma(v_this, pf);
  };

  f32x16 sa[NT], sb[NT];
  if (blk0 < blk1) {
    issue(kc, blk0, kst(blk0));
    issue(vc, blk0, vst(blk0));
    attn_wait_loads();
    attn_barrier();
    if (blk0 + 1 < blk1) issue(kc, blk0 + 1, kst(blk0 + 1));
    s_mfma(kst(blk0), sa);
  }
  int blk = blk0;
  for (; blk + 1 < blk1; blk += 2) {
    iteration(std::integral_constant<int, 0>(), blk, sa, sb);
    iteration(std::integral_constant<int, 1>(), blk + 1, sb, sa);
  }
  if (blk < blk1) iteration(std::integral_constant<int, 0>(), blk, sa, sb);
  attn_wait_loads();  // no direct load may still be writing LDS when the workgroup ends

  if (Z > 1) {  // unnormalised partial of this key split
    if (qok) {
      const int64_t r = ((int64_t)z * T + qi) * nq + h;
      float* dst = part_acc + r * HD;
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) dst[32 * d + 8 * (v >> 2) + 4 * half_sel + (v & 3)] = o[d][v];
      if (half_sel == 0) {
        part_ml[r * 2] = m_run;
        part_ml[r * 2 + 1] = l_run;
      }
    }
    return;
  }
  if (qok) {
    const float inv = 1.0f / l_run;
    uint16_t* dst = out + ((int64_t)qi * nq + h) * HD;
    bool bad = false;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        dst[32 * d + 8 * (v >> 2) + 4 * half_sel + (v & 3)] = f16_checked(o[d][v] * inv, bad);
    raise_err(err_flag, bad, kErrF16Range);
  }
}

// Merge of Z key splits: o[q][h][d] = sum_z 2^(m_z - M) acc_z[d] / sum_z 2^(m_z - M) l_z
// (a split without keys has m = -inf, l = 0 and weight 0).  One thread per 4 dims;
// the (max, sum) pairs and vectors of the first four splits are requested together,
// so the merge takes one memory round trip (70B-shaped attention with its merge
// 97.0 -> 93.5 us per layer).
template <int HD>
__global__ __launch_bounds__(256) void attn_prefill_combine_kernel(const float* part_acc, const float* part_ml,
                                                                   uint16_t* out, int rows, int Z, int* err_flag) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;  // over rows * HD/4
  if (e >= (int64_t)rows * (HD / 4)) return;
  const int64_t r = e / (HD / 4);
  const int d4 = (int)(e % (HD / 4));
  constexpr int ZP = 4;  // splits whose (max, sum) and vector are requested together
  float2 mlp[ZP];
  v4f ap[ZP];
#pragma unroll
  for (int z = 0; z < ZP; ++z) {
    const int zz = z < Z ? z : 0;
    mlp[z] = reinterpret_cast<const float2*>(part_ml)[(int64_t)zz * rows + r];
    ap[z] = reinterpret_cast<const v4f*>(part_acc + ((int64_t)zz * rows + r) * HD)[d4];
  }
  float M = -INFINITY;
#pragma unroll
  for (int z = 0; z < ZP; ++z)
    if (z < Z && mlp[z].y > 0.f) M = fmaxf(M, mlp[z].x);
  for (int z = ZP; z < Z; ++z) {
    const float m = part_ml[((int64_t)z * rows + r) * 2], l = part_ml[((int64_t)z * rows + r) * 2 + 1];
    if (l > 0.f) M = fmaxf(M, m);
  }
  v4f acc = {0.f, 0.f, 0.f, 0.f};
  float L = 0.f;
#pragma unroll
  for (int z = 0; z < ZP; ++z) {
    const float w = z < Z && mlp[z].y > 0.f ? exp2f(mlp[z].x - M) : 0.f;
    acc += w * ap[z];
    L += w * mlp[z].y;
  }
  for (int z = ZP; z < Z; ++z) {
    const float m = part_ml[((int64_t)z * rows + r) * 2], l = part_ml[((int64_t)z * rows + r) * 2 + 1];
    const float w = l > 0.f ? exp2f(m - M) : 0.f;
    acc += w * reinterpret_cast<const v4f*>(part_acc + ((int64_t)z * rows + r) * HD)[d4];
    L += w * l;
  }
  acc *= 1.0f / L;
  bool bad = false;
  reinterpret_cast<uint2*>(out + r * HD)[d4] =
      uint2{pack_f16_checked(acc.x, acc.y, bad), pack_f16_checked(acc.z, acc.w, bad)};
  raise_err(err_flag, bad, kErrF16Range);
}

// ------------------------------------------------------------------ final copy
// Hidden output of the stage: the residual stream plus the nsplit pending
// split-K slices of the last down projection (slice stride n).
__global__ void store_rows_kernel(const float* x, const float* part, int nsplit, void* out, int out_bf16,
                                  int64_t n) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= n) return;
  float v = x[i];
  for (int sl = 0; sl < nsplit; ++sl) v += part[sl * n + i];
  if (out_bf16) reinterpret_cast<uint16_t*>(out)[i] = to_bf16(v);
  else reinterpret_cast<float*>(out)[i] = v;
}

// ------------------------------------------------------------------ host side
static int64_t a256(int64_t n) { return (n + 255) & ~(int64_t)255; }

void prefill_free(PrefillWorkspace& ws) {
  if (ws.mem) (void)hipFree(ws.mem);
  ws = PrefillWorkspace{};
}

// Bytes of each workspace buffer for a chunk of a.T tokens, in layout order:
// x, xn, part, q, o, act.
static void prefill_sizes(const PrefillArgs& a, int64_t (&sz)[6]) {
  const int64_t T = a.T, H = a.H, nqkv = (int64_t)(a.nq + 2 * a.nkv) * a.hd;
  // the split-K slices of the largest of the QKV, O and down projections
  const int64_t part_qkv = (int64_t)gemm_splitk(a.T, (int)nqkv, H) * T * nqkv;
  const int64_t part_o = (int64_t)gemm_splitk(a.T, H, a.nq * a.hd) * T * H;
  const int64_t part_d = (int64_t)gemm_splitk(a.T, H, a.F) * T * H;
  const int64_t part_attn = (int64_t)KF_PF_ATTN_SPLIT * T * a.nq * (a.hd + 2);  // key-split attention partials
  const int64_t part = std::max(std::max(part_qkv, part_attn), std::max(part_o, part_d));
  sz[0] = a256(T * H * 4);
  sz[1] = a256(T * H * 2);
  sz[2] = a256(part * 4);
  sz[3] = a256(T * a.nq * a.hd * 2);
  sz[4] = a256(T * a.nq * a.hd * 2);
  sz[5] = a256(T * a.F * 2);
}

int64_t prefill_ws_bytes(const PrefillArgs& a) {
  int64_t sz[6];
  prefill_sizes(a, sz);
  return sz[0] + sz[1] + sz[2] + sz[3] + sz[4] + sz[5];
}

void prefill_carve(PrefillWorkspace& ws, char* base, const PrefillArgs& a) {
  int64_t sz[6];
  prefill_sizes(a, sz);
  char* p = base;
  ws.x = (float*)p;
  p += sz[0];
  ws.xn = (uint16_t*)p;
  p += sz[1];
  ws.part = (float*)p;
  p += sz[2];
  ws.q = (uint16_t*)p;
  p += sz[3];
  ws.o = (uint16_t*)p;
  p += sz[4];
  ws.act = (uint16_t*)p;
  ws.pending = 0;
}

hipError_t prefill_reserve(PrefillWorkspace& ws, const PrefillArgs& a) {
  if (a.T <= ws.cap_T && ws.mem) return hipSuccess;
  const int64_t total = prefill_ws_bytes(a);
  char* mem = nullptr;
  // Drain work that may still use the old buffer before freeing it.
  hipError_t e = hipStreamSynchronize(a.stream);
  if (e != hipSuccess) return e;
  e = hipMalloc((void**)&mem, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return hipErrorOutOfMemory;
  }
  prefill_free(ws);
  ws.mem = mem;
  ws.cap_T = a.T;
  prefill_carve(ws, mem, a);
  return hipSuccess;
}

hipError_t prefill_layer(PrefillWorkspace& ws, const PrefillArgs& a, const PrefillLayer& l, const Tracer& tr) {
  hipStream_t s = a.stream;
  const int T = a.T, H = a.H, nqkv = (a.nq + 2 * a.nkv) * a.hd;
  const int64_t TH = (int64_t)T * H;
  hipError_t e;
  // Class ids follow kf_kernel_class of the public header.
  enum { NORM = 8, QKV = 9, ROPE = 10, ATTN = 11, OPROJ = 12, GATEUP = 13, DOWN = 14, STORE = 15 };
  // The previous layer's down projection may still be pending as split-K slices.
  tr.begin(NORM);
  hipLaunchKernelGGL(rmsnorm_rows_f16_kernel, dim3(T), dim3(256), 0, s, ws.x, ws.part, ws.pending, TH, l.g_attn,
                     a.eps, ws.xn, H, a.err_flag);
  tr.end(NORM);
  ws.pending = 0;
  if ((e = hipGetLastError()) != hipSuccess) return e;
  tr.begin(QKV);
  const int s_qkv = gemm_splitk(T, nqkv, H);
  if (s_qkv > kMaxSlices || gemm_splitk(T, H, a.nq * a.hd) > kMaxSlices || gemm_splitk(T, H, a.F) > kMaxSlices)
    return hipErrorInvalidValue;  // more split-K slices than the consuming kernels add
  e = launch_gemm(kGemmPartialF32, ws.xn, l.wqkv, nullptr, T, nqkv, H, ws.part, nullptr, a.err_flag, s);
  tr.end(QKV);
  if (e != hipSuccess) return e;
  tr.begin(ROPE);
  hipLaunchKernelGGL(rope_kv_kernel, dim3(T), dim3(256), 0, s, ws.part, s_qkv, (int64_t)T * nqkv, ws.q, l.kc, l.vc,
                     a.kv, a.user, a.rope_cos, a.rope_sin, a.nq, a.nkv, a.hd, a.pos0, l.g_qn, l.g_kn, a.eps,
                     a.err_flag);
  tr.end(ROPE);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const float sl2 = (float)(1.4426950408889634 / std::sqrt((double)a.hd));
  // Key splits: enough workgroups for two per CU when the chunk alone gives fewer.
  const int qtiles = (T + 127) / 128;
  const int Z = qtiles * a.nq >= 512 ? 1 : KF_PF_ATTN_SPLIT;
  const dim3 ag(qtiles, a.nq, Z);
  float* pacc = ws.part;
  float* pml = ws.part + (int64_t)Z * T * a.nq * a.hd;
  tr.begin(ATTN);
  if (a.hd == 128)
    hipLaunchKernelGGL(attn_prefill_kernel<128>, ag, dim3(256), 0, s, ws.q, l.kc, l.vc, a.kv, a.user, ws.o, pacc,
                       pml, T, a.nq, a.nkv, a.pos0, sl2, a.err_flag);
  else if (a.hd == 64)
    hipLaunchKernelGGL(attn_prefill_kernel<64>, ag, dim3(256), 0, s, ws.q, l.kc, l.vc, a.kv, a.user, ws.o, pacc,
                       pml, T, a.nq, a.nkv, a.pos0, sl2, a.err_flag);
  else
    return hipErrorInvalidValue;
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (Z > 1) {
    const int rows = T * a.nq;
    const int64_t n = (int64_t)rows * (a.hd / 4);
    const dim3 cg((unsigned)((n + 255) / 256));
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_prefill_combine_kernel<128>, cg, dim3(256), 0, s, pacc, pml, ws.o, rows, Z, a.err_flag);
    else
      hipLaunchKernelGGL(attn_prefill_combine_kernel<64>, cg, dim3(256), 0, s, pacc, pml, ws.o, rows, Z, a.err_flag);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  tr.end(ATTN);
  // O and down: split along K into slices that the next norm (or the output
  // store) adds in order; an unsplit projection adds into x directly.
  auto resid_proj = [&](int cls, const uint16_t* A, const uint16_t* W, int K, int* pend) {
    const int sp = gemm_splitk(T, H, K);
    tr.begin(cls);
    const hipError_t le = sp > 1 ? launch_gemm(kGemmPartialF32, A, W, nullptr, T, H, K, ws.part, nullptr, a.err_flag, s)
                                 : launch_gemm(kGemmResidF32, A, W, nullptr, T, H, K, ws.x, nullptr, a.err_flag, s);
    tr.end(cls);
    *pend = sp > 1 ? sp : 0;
    return le;
  };
  int pend_o = 0;
  if ((e = resid_proj(OPROJ, ws.o, l.wo, a.nq * a.hd, &pend_o)) != hipSuccess) return e;
  tr.begin(NORM);
  hipLaunchKernelGGL(rmsnorm_rows_f16_kernel, dim3(T), dim3(256), 0, s, ws.x, ws.part, pend_o, TH, l.g_mlp, a.eps,
                     ws.xn, H, a.err_flag);
  tr.end(NORM);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  tr.begin(GATEUP);
  e = launch_gemm(kGemmSwiGLU, ws.xn, l.wg, l.wu, T, 2 * a.F, H, nullptr, ws.act, a.err_flag, s);
  tr.end(GATEUP);
  if (e != hipSuccess) return e;
  if ((e = resid_proj(DOWN, ws.act, l.wd, a.F, &ws.pending)) != hipSuccess) return e;
  if (l.out) {
    tr.begin(STORE);
    hipLaunchKernelGGL(store_rows_kernel, dim3((unsigned)((TH + 255) / 256)), dim3(256), 0, s, ws.x, ws.part,
                       ws.pending, l.out, l.out_bf16, TH);
    tr.end(STORE);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kf

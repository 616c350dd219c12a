// Prefill projections on the matrix cores: C[M][N] (+)= A[M][K] x W[N][K]^T.
//
// A is fp16 activations, W is fp16 weights (converted from the model's bf16
// once, when the stage is created), both K-contiguous; the product runs on v_mfma_f32_32x32x16_f16 with
// fp32 accumulation.  At a 512-token chunk the projections are large enough
// to be bound by the matrix cores, which sets the tile shape:
//   * 256 x 256 x 32 workgroup tiles, eight waves (two per SIMD) of 128 x 64,
//     8 accumulator blocks each: per K step a wave reads 12 KB of fragments
//     from LDS for 16 MFMAs.  Two waves per SIMD let one issue MFMAs while the
//     other waits on LDS or the barrier (measured 4% faster than four waves of
//     128 x 128 with 16 blocks each, which remains selectable);
//   * operands go from global memory straight into a 4-stage LDS ring with
//     global_load_lds (no register staging), so loads run three to four K
//     steps (1.3 - 1.7 us of math at full rate) ahead; chunks are XOR-swizzled
//     within a row so that fragment reads are free of bank conflicts;
//   * each wave reads the fragments of the next 16-wide K slice while the
//     MFMAs of the current one run;
//   * narrow projections (few 256-wide column tiles) are split along K over
//     several workgroups so that the grid covers the 256 CUs; the slices are
//     stored whole for the consuming kernel to add in order (kGemmPartialF32).
// Operand fragment layout of v_mfma_f32_32x32x16_f16 (lane l of 64):
//   A: row l%32, k = 8*(l/32) .. +7      B: column l%32, k = 8*(l/32) .. +7
//   D: element v (0..15) at row 8*(v/4) + 4*(l/32) + v%4, column l%32
#include "kernels.h"
#include "prefill.h"

namespace kf {
namespace {

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int BM = 256, BN = 256, BK = 32;
#ifndef KF_GEMM_WN
#define KF_GEMM_WN 4
#endif
// Waves along N: 2 gives four waves of 128 x 128 (one per SIMD), 4 gives eight
// waves of 128 x 64 (two per SIMD, half the accumulators each).
constexpr int kGemmWN = KF_GEMM_WN;
constexpr int kGemmThreads = 128 * kGemmWN;
#ifndef KF_GEMM_READS_PER_SLOT
#define KF_GEMM_READS_PER_SLOT 1  // fragment reads issued per MFMA slot
#endif
#ifndef KF_GEMM_SPLIT_FLOOR
#define KF_GEMM_SPLIT_FLOOR 1  // K slices per tile: floor (1) or ceiling (0) of 256 / tiles
#endif
#ifndef KF_GEMM_STAGES
#define KF_GEMM_STAGES 4
#endif
constexpr int STAGES = KF_GEMM_STAGES;      // LDS ring depth: loads run up to STAGES K steps ahead
static_assert(STAGES >= 3 && STAGES <= 5, "ring depth");
constexpr int TILE_BYTES = BM * BK * 2;     // one operand's tile per stage (16 KB)
constexpr int ROW_BYTES = BK * 2;           // 64 B: four 16-byte chunks per tile row

__device__ __forceinline__ f32x16 mfma32(v4u a, v4u b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

// Chunk c (0..3) of tile row r is stored at slot c ^ f(r) of that row, with
// f(r) = (r/2 ^ r/4) % 4: any 8 consecutive rows hit distinct 16-byte bank
// groups of a 32-bank LDS, and any 16 consecutive rows of a 64-bank one, so
// the fragment reads (one row per lane) are free of bank conflicts.
__device__ __forceinline__ int swz(int r, int c) { return c ^ (((r >> 1) ^ (r >> 2)) & 3); }

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// Wait until this wave's LDS reads have returned (global loads may stay in flight).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14)); }

// Workgroup barrier that orders LDS accesses without waiting on outstanding
// global loads (the compiler may not move memory operations across it).
__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

struct Params {
  const uint16_t* A;
  const uint16_t* W;
  const uint16_t* W2;
  int M, N, K;
  int splitk;  // K slices (1: read-modify-write or SwiGLU epilogue)
  float* C;
  uint16_t* Cb;
  int* err_flag;
};

template <int EPI>
__global__ __launch_bounds__(kGemmThreads) void gemm256_kernel(const Params p) {
  constexpr int WN = kGemmWN;
  constexpr int NW = 2 * WN;                 // waves
  constexpr int JW = 8 / WN;                 // 32-column blocks per wave (128 / 64 columns)
  constexpr int LOADS = TILE_BYTES / 1024 / NW;  // 1 KB direct loads per wave per operand per stage
  constexpr int SLOTS = 4 * JW;              // MFMAs per wave per 16-wide K slice
  static_assert(WN == 2 || WN == 4, "four or eight waves");
  // STAGES x (A tile, W tile), each [256 rows][4 swizzled 16-byte chunks]; both fp16.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * 2 * TILE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;  // 2 x WN waves of 128 x (256 / WN)
  const int mt = (p.M + BM - 1) / BM, nt = (p.N + BN - 1) / BN, ntiles = mt * nt;
  const int nwg = ntiles * p.splitk;
  // Tiles sharing a weight panel (same column tile) go to the same XCD, where
  // they reuse it through that XCD's L2 (workgroups are dealt round-robin).
  int bid = blockIdx.x;
  if (nwg % 8 == 0) bid = (bid % 8) * (nwg / 8) + bid / 8;
  const int ks = bid % p.splitk, t = bid / p.splitk;
  const int tm = t % mt, tn = t / mt;
  const int m0 = tm * BM, n0 = tn * BN;
  const int K = p.K;
  const int nk_all = K / BK;
  const int k_begin = (int)((int64_t)nk_all * ks / p.splitk), k_end = (int)((int64_t)nk_all * (ks + 1) / p.splitk);
  const int nk = k_end - k_begin;

  // Direct global -> LDS loads: load j of this wave fills tile rows
  // 16 (NW j + wave) .. +15; lane l writes row 16 (NW j + wave) + l/4, slot l%4,
  // so it fetches the chunk that belongs in that slot.
  const int w_rows = EPI == kGemmSwiGLU ? (p.N >> 1) : p.N;
  const uint16_t* asrc[LOADS];
  const uint16_t* wsrc[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int r = 16 * (NW * j + wave) + (lane >> 2);
    const int c = swz(r, lane & 3);
    const int ar = m0 + r < p.M ? m0 + r : p.M - 1;  // rows past M load a valid row; they are never stored
    asrc[j] = p.A + (int64_t)ar * K + (int64_t)k_begin * BK + c * 8;
    // weight tile row r: for SwiGLU, 32-row groups alternate gate / up rows of the same outputs
    int wr;
    const uint16_t* wb;
    if (EPI == kGemmSwiGLU) {
      wr = (n0 >> 1) + (r >> 6) * 32 + (r & 31);
      wb = ((r >> 5) & 1) ? p.W2 : p.W;
    } else {
      wr = n0 + r;
      wb = p.W;
    }
    if (wr >= w_rows) wr = w_rows - 1;  // columns past N load a valid row; they are never stored
    wsrc[j] = wb + (int64_t)wr * K + (int64_t)k_begin * BK + c * 8;
  }
  auto issue = [&](int kt, int stage) {
    uint8_t* abuf = smem + stage * 2 * TILE_BYTES;
    uint8_t* wbuf = abuf + TILE_BYTES;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      __builtin_amdgcn_global_load_lds(asrc[j] + (int64_t)kt * BK, (lds_ptr)(abuf + 1024 * (NW * j + wave)), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(wsrc[j] + (int64_t)kt * BK, (lds_ptr)(wbuf + 1024 * (NW * j + wave)), 16, 0, 0);
    }
  };

  f32x16 acc[4][JW];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < JW; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // The K loop is scheduled by hand: each half step is SLOTS MFMA slots; the
  // first slots also issue the fragment reads for the next half (and, after
  // the barrier, one global->LDS load each).
  const int rl = lane & 31, kh = lane >> 5;
  // fragment read q (0..JW+3) of sub-step s (16 values of K) of a stage: weight
  // block q for q < JW, then A block q-JW
  auto read_frag = [&](int stage, int s, int q, v4u (&fa)[4], v4u (&fw)[JW]) {
    const bool w = q < JW;
    const uint8_t* buf = smem + stage * 2 * TILE_BYTES + (w ? TILE_BYTES : 0);
    const int r = w ? wn * (32 * JW) + 32 * q + rl : wm * 128 + 32 * (q - JW) + rl;
    const v4u v = *reinterpret_cast<const v4u*>(buf + r * ROW_BYTES + swz(r, 2 * s + kh) * 16);
    if (w) fw[q] = v;
    else fa[q - JW] = v;
  };
  // global->LDS load q (0..2 LOADS - 1) of step kt into a stage: A for even q, W for odd q
  auto load_part = [&](int kt, int stage, int q) {
    uint8_t* buf = smem + stage * 2 * TILE_BYTES + (q & 1) * TILE_BYTES + 1024 * (NW * (q >> 1) + wave);
    const uint16_t* src = ((q & 1) ? wsrc[q >> 1] : asrc[q >> 1]) + (int64_t)kt * BK;
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)buf, 16, 0, 0);
  };
  // One half step: the SLOTS MFMAs on (fa, fw), the reads of the next fragments
  // into (na, nw), RPS per slot from slot 0, and optionally the loads of step kt.
  auto half = [&](const v4u (&fa)[4], const v4u (&fw)[JW], int rstage, int rs, v4u (&na)[4], v4u (&nw)[JW],
                  bool load, int kt, int lstage) {
    constexpr int RPS = KF_GEMM_READS_PER_SLOT;
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) {
      acc[q / JW][q % JW] = mfma32(fa[q / JW], fw[q % JW], acc[q / JW][q % JW]);
#pragma unroll
      for (int r = 0; r < RPS; ++r)
        if (q * RPS + r < JW + 4) read_frag(rstage, rs, q * RPS + r, na, nw);
      if (load && q < 2 * LOADS) load_part(kt, lstage, q);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Ring: step k lives in stage k % STAGES.  The fragments of sub-step s+1 are
  // read while the MFMAs of sub-step s run.  The barrier in the middle of step
  // k releases step k+1's data to every wave and hands stage k % STAGES (whose
  // last reads were in step k's first half) to the loads of step k + STAGES.
  // Past the last step those loads repeat step nk-1 into stages that are not
  // read again, which keeps the loop free of branches and the wait counts fixed.
#pragma unroll
  for (int s = 0; s < STAGES; ++s) issue(s < nk ? s : nk - 1, s);
  wait_vm<(STAGES - 1) * 2 * LOADS>();  // step 0 has landed
  block_barrier();
  v4u fa0[4], fw0[JW], fa1[4], fw1[JW];
#pragma unroll
  for (int q = 0; q < JW + 4; ++q) read_frag(0, 0, q, fa0, fw0);
  for (int k = 0; k + 1 < nk; ++k) {
    __builtin_amdgcn_sched_barrier(0);
    half(fa0, fw0, k % STAGES, 1, fa1, fw1, false, 0, 0);
    // this wave's loads for step k+1 are complete once only the next STAGES-2 steps' remain
    wait_vm<(STAGES - 2) * 2 * LOADS>();
    wait_lds();  // this wave's reads of stage k % STAGES have returned (issued a half step ago)
    // Every wave's loads for step k+1 have landed and every wave's reads of
    // stage k % STAGES have returned.  A bare barrier: a fence here would also
    // drain the loads in flight.
    block_barrier();
    half(fa1, fw1, (k + 1) % STAGES, 0, fa0, fw0, true, k + STAGES < nk ? k + STAGES : nk - 1, k % STAGES);
  }
  {
    const int k = nk - 1;
    half(fa0, fw0, k % STAGES, 1, fa1, fw1, false, 0, 0);
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) acc[q / JW][q % JW] = mfma32(fa1[q / JW], fw1[q % JW], acc[q / JW][q % JW]);
  }
  wait_vm<0>();  // no load may still be writing LDS when the workgroup ends

  // Epilogue.
  const int rq = 4 * (lane >> 5);
  bool bad = false;  // an fp16 SwiGLU output out of range
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = m0 + wm * 128 + 32 * i + 8 * (v >> 2) + rq + (v & 3);
      if (row >= p.M) continue;
      if (EPI == kGemmSwiGLU) {
#pragma unroll
        for (int jj = 0; jj < JW / 2; ++jj) {  // blocks (2jj, 2jj+1) are gate / up of the same outputs
          const int j = (n0 >> 1) + wn * (16 * JW) + 32 * jj + rl;
          if (j < (p.N >> 1)) {
            const float g = acc[i][2 * jj][v], u = acc[i][2 * jj + 1][v];
            p.Cb[(int64_t)row * (p.N >> 1) + j] = f16_checked(g / (1.0f + expf(-g)) * u, bad);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < JW; ++j) {
          const int col = n0 + wn * (32 * JW) + 32 * j + rl;
          if (col >= p.N) continue;
          float* c = p.C + (int64_t)row * p.N + col;
          if (EPI == kGemmResidF32) *c += acc[i][j][v];
          else c[(int64_t)ks * p.M * p.N] = acc[i][j][v];
        }
      }
    }
  }
  if (EPI == kGemmSwiGLU) raise_err(p.err_flag, bad, kErrF16Range);
}

}  // namespace

#ifndef KF_GEMM_MAX_SPLIT
#define KF_GEMM_MAX_SPLIT 8  // upper bound on K slices per output tile
#endif

int gemm_splitk(int M, int N, int K) {
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int nk = K / BK;
  if (tiles >= 192 || nk < 128) return 1;  // enough tiles, or a short (cheap) reduction
  int s = KF_GEMM_SPLIT_FLOOR ? 256 / tiles : (256 + tiles - 1) / tiles;
  if (s > nk / 64) s = nk / 64;  // keep at least 64 K steps per slice
  if (s > KF_GEMM_MAX_SPLIT) s = KF_GEMM_MAX_SPLIT;
  return s < 1 ? 1 : s;
}

hipError_t launch_gemm(int epi, const uint16_t* A, const uint16_t* W, const uint16_t* W2, int M, int N, int K,
                       float* C, uint16_t* Cb, int* err_flag, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0 || K % BK) return hipErrorInvalidValue;
  if (epi == kGemmSwiGLU && N % 2) return hipErrorInvalidValue;
  // the nonlinearity and the residual update need complete sums: only the partial epilogue splits K
  Params p{A, W, W2, M, N, K, epi == kGemmPartialF32 ? gemm_splitk(M, N, K) : 1, C, Cb, err_flag};
  const int grid = ((M + BM - 1) / BM) * ((N + BN - 1) / BN) * p.splitk;
  switch (epi) {
    case kGemmResidF32: hipLaunchKernelGGL(gemm256_kernel<kGemmResidF32>, dim3(grid), dim3(kGemmThreads), 0, s, p); break;
    case kGemmSwiGLU: hipLaunchKernelGGL(gemm256_kernel<kGemmSwiGLU>, dim3(grid), dim3(kGemmThreads), 0, s, p); break;
    case kGemmPartialF32: hipLaunchKernelGGL(gemm256_kernel<kGemmPartialF32>, dim3(grid), dim3(kGemmThreads), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kf

// Prefill projections on the matrix cores: C[M][N] (+)= A[M][K] x W[N][K]^T.
//
// A is fp16 activations, W is fp16 weights (converted from the model's bf16
// once, when the stage is created), both K-contiguous; the product runs on v_mfma_f32_32x32x16_f16 with
// fp32 accumulation.  At a 512-token chunk the projections are large enough
// to be bound by the matrix cores, which sets the tile shape:
//   * 256 x 256 x 64 workgroup tiles, eight waves (two per SIMD) of 128 x 64,
//     8 accumulator blocks each: per K step a wave reads 24 KB of fragments
//     from LDS for 32 MFMAs.  Two waves per SIMD let one issue MFMAs while the
//     other waits on LDS or the barrier (measured 4% faster than four waves of
//     128 x 128 with 16 blocks each, which remains selectable);
//   * operands go from global memory straight into LDS rings with
//     global_load_lds (no register staging).  A 64-deep K step makes each load
//     instruction fetch 8 rows x 128 B, i.e. whole cache lines; 32-deep steps
//     fetched 16 half lines per instruction and ran the 70B gate/up shape
//     5-7% slower.  The weights, which stream from HBM, get a 3-stage ring
//     (loads run two K steps ahead), the activations, which stay in L2, a
//     2-stage one: 160 KB together, 2% faster on that shape than 2 stages of
//     both (the whole 70B chunk 1%, the Qwen3-32B-shaped one 2.5%);
//   * chunks are XOR-swizzled within a row so that fragment reads are free of
//     bank conflicts;
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

#ifndef KF_GEMM_BK
#define KF_GEMM_BK 64
#endif
constexpr int BM = 256, BN = 256, BK = KF_GEMM_BK;
static_assert(BK == 32 || BK == 64, "K step");
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
#define KF_GEMM_STAGES (BK == 32 ? 4 : 2)
#endif
#ifndef KF_GEMM_WSTAGES
#define KF_GEMM_WSTAGES (BK == 32 ? 4 : 3)
#endif
// LDS ring depths: activation loads run up to SA K steps ahead, weight loads up to SW.
constexpr int SA = KF_GEMM_STAGES, SW = KF_GEMM_WSTAGES;
constexpr int TILE_BYTES = BM * BK * 2;     // one operand's tile per stage (16 or 32 KB)
constexpr int ROW_BYTES = BK * 2;           // 64 or 128 B per tile row
constexpr int CH = BK / 8;                  // 16-byte chunks per tile row
constexpr int SS = BK / 16;                 // 16-wide K slices (MFMA steps) per K step
static_assert(SA >= 2 && SW >= SA && SW <= SA + 1 && (SA + SW) * TILE_BYTES <= 160 * 1024, "ring depths");

__device__ __forceinline__ f32x16 mfma32(v4u a, v4u b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

// Chunk c of tile row r is stored at slot c ^ f(r) of that row.  Four chunks
// per row: f(r) = (r/2 ^ r/4) % 4; eight: f(r) = r % 8 ^ (r/8) % 2.  Either way
// any 8 consecutive rows hit distinct 16-byte bank groups of a 32-bank LDS,
// and any 16 consecutive rows of a 64-bank one, so the fragment reads (one
// row per lane) are free of bank conflicts.
__device__ __forceinline__ int swz(int r, int c) {
  return CH == 4 ? c ^ (((r >> 1) ^ (r >> 2)) & 3) : c ^ ((r & 7) ^ ((r >> 3) & 1));
}

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
  // SA A tiles, then SW W tiles, each [256 rows][CH swizzled 16-byte chunks]; both fp16.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[(SA + SW) * TILE_BYTES];

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

  // Direct global -> LDS loads: load j of this wave fills the 1 KB of tile rows
  // (64 / CH) (NW j + wave) .. + 64 / CH - 1; lane l writes row
  // (64 / CH) (NW j + wave) + l / CH, slot l % CH, so it fetches the chunk that
  // belongs in that slot (the CH lanes of a row cover ROW_BYTES contiguous bytes).
  const int w_rows = EPI == kGemmSwiGLU ? (p.N >> 1) : p.N;
  const uint16_t* asrc[LOADS];
  const uint16_t* wsrc[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int r = (64 / CH) * (NW * j + wave) + lane / CH;
    const int c = swz(r, lane % CH);
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
  // Step kt's stages; past the last step a load fetches step nk-1 again (into
  // the stage of the step it stands in for, which is never read).
  auto abuf = [&](int kt) { return smem + (kt % SA) * TILE_BYTES; };
  auto wbuf = [&](int kt) { return smem + (SA + kt % SW) * TILE_BYTES; };
  auto src_step = [&](int kt) { return (int64_t)(kt < nk ? kt : nk - 1) * BK; };
  auto issue_a = [&](int kt) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      // (named operands: the host pass drops the kernel's launch stub when the
      // builtin's pointer argument is a call expression)
      const uint16_t* src = asrc[j] + src_step(kt);
      uint8_t* dst = abuf(kt) + 1024 * (NW * j + wave);
      __builtin_amdgcn_global_load_lds(src, (lds_ptr)dst, 16, 0, 0);
    }
  };
  auto issue_w = [&](int kt) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const uint16_t* src = wsrc[j] + src_step(kt);
      uint8_t* dst = wbuf(kt) + 1024 * (NW * j + wave);
      __builtin_amdgcn_global_load_lds(src, (lds_ptr)dst, 16, 0, 0);
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
  // fragment read q (0..JW+3) of slice s (16 values of K) of step k: weight
  // block q for q < JW, then A block q-JW
  auto read_frag = [&](int k, int s, int q, v4u (&fa)[4], v4u (&fw)[JW]) {
    const bool w = q < JW;
    const uint8_t* buf = w ? wbuf(k) : abuf(k);
    const int r = w ? wn * (32 * JW) + 32 * q + rl : wm * 128 + 32 * (q - JW) + rl;
    const v4u v = *reinterpret_cast<const v4u*>(buf + r * ROW_BYTES + swz(r, 2 * s + kh) * 16);
    if (w) fw[q] = v;
    else fa[q - JW] = v;
  };
  // global->LDS load q (0..2 LOADS - 1): A of step ka for q < LOADS, then W of step kw
  auto load_part = [&](int ka, int kw, int q) {
    const bool w = q >= LOADS;
    const int j = w ? q - LOADS : q;
    uint8_t* buf = (w ? wbuf(kw) : abuf(ka)) + 1024 * (NW * j + wave);
    const uint16_t* src = w ? wsrc[j] + src_step(kw) : asrc[j] + src_step(ka);
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)buf, 16, 0, 0);
  };
  // One slice: the SLOTS MFMAs on (fa, fw), the reads of the next fragments
  // (slice rs of step rk) into (na, nw), RPS per slot from slot 0, and
  // optionally the loads of steps ka (A) and kw (W).
  auto half = [&](const v4u (&fa)[4], const v4u (&fw)[JW], int rk, int rs, v4u (&na)[4], v4u (&nw)[JW],
                  bool load, int ka, int kw) {
    constexpr int RPS = KF_GEMM_READS_PER_SLOT;
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) {
      acc[q / JW][q % JW] = mfma32(fa[q / JW], fw[q % JW], acc[q / JW][q % JW]);
#pragma unroll
      for (int r = 0; r < RPS; ++r)
        if (q * RPS + r < JW + 4) read_frag(rk, rs, q * RPS + r, na, nw);
      if (load && q < 2 * LOADS) load_part(ka, kw, q);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Rings: step k's activations live in A stage k % SA, its weights in W
  // stage k % SW.  The fragments of slice s+1 are read while the MFMAs of
  // slice s run.  The barrier before the last slice of step k releases step
  // k+1's data to every wave and hands both of step k's stages (whose last
  // reads were issued in the slice before) to the loads of step k + SA (A) and
  // k + SW (W), which are issued A first.  Past the last step those loads
  // repeat step nk-1 into stages that are not read again, which keeps the loop
  // free of branches and the wait counts fixed.
#pragma unroll
  for (int s = 0; s < SW; ++s) {
    if (s < SA) issue_a(s);
    issue_w(s);
  }
  wait_vm<(SA + SW - 2) * LOADS>();  // step 0 has landed
  block_barrier();
  v4u fa[2][4], fw[2][JW];
#pragma unroll
  for (int q = 0; q < JW + 4; ++q) read_frag(0, 0, q, fa[0], fw[0]);
  static_assert(SS % 2 == 0, "a step starts with its fragments in buffer 0");
  for (int k = 0; k + 1 < nk; ++k) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s + 1 < SS; ++s)
      half(fa[s & 1], fw[s & 1], k, s + 1, fa[(s + 1) & 1], fw[(s + 1) & 1], false, 0, 0);
    // This wave's loads for step k+1 are complete once only later steps' remain
    // in flight: the A loads of steps k+2 .. k+SA-1 and the W loads of steps
    // k+2 .. k+SW-1, which are the most recent (SA - 2) * 2 + (SW - SA) groups.
    wait_vm<((SA - 2) * 2 + (SW - SA)) * LOADS>();
    wait_lds();  // this wave's reads of step k's stages have returned (issued a slice ago)
    // Every wave's loads for step k+1 have landed and every wave's reads of
    // step k's stages have returned.  A bare barrier: a fence here would also
    // drain the loads in flight.
    block_barrier();
    half(fa[1], fw[1], k + 1, 0, fa[0], fw[0], true, k + SA, k + SW);
  }
  {
    const int k = nk - 1;
#pragma unroll
    for (int s = 0; s + 1 < SS; ++s)
      half(fa[s & 1], fw[s & 1], k, s + 1, fa[(s + 1) & 1], fw[(s + 1) & 1], false, 0, 0);
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) acc[q / JW][q % JW] = mfma32(fa[1][q / JW], fw[1][q % JW], acc[q / JW][q % JW]);
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
  const int k32 = K / 32;
  if (tiles >= 192 || k32 < 128) return 1;  // enough tiles, or a short (cheap) reduction
  int s = KF_GEMM_SPLIT_FLOOR ? 256 / tiles : (256 + tiles - 1) / tiles;
  if (s > k32 / 64) s = k32 / 64;  // keep at least 2048 of K per slice
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

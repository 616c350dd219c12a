// Prefill projections on the matrix cores: C[M][N] (+)= A[M][K] x W[N][K]^T.
//
// A is fp16 activations, W is fp16 weights (converted from the model's bf16
// once, when the stage is created), both K-contiguous; the product runs on v_mfma_f32_32x32x16_f16 with
// fp32 accumulation.  At a 512-token chunk the projections are large enough
// to be bound by the matrix cores, which sets the tile shape:
//   * 256 x 256 x 64 workgroup tiles, eight waves (two per SIMD) of 128 x 64,
//     8 accumulator blocks each: per K step a wave reads 24 KB of fragments
//     from LDS for 32 MFMAs.  Two waves per SIMD let one issue MFMAs while the
//     other waits on LDS or the barrier (four waves of 128 x 128 measured 4-5%
//     slower);
//   * the SwiGLU projection takes 256 x 224 tiles when they fill whole rounds
//     of the 256 CUs in fewer tile-times (the 70B gate/up shape: 512 tiles in
//     2 rounds, against 448 of 256 x 256 whose second round is three quarters
//     full): eight waves of 64 x 128 and 64 x 96, one of each per SIMD;
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
constexpr int kGemmThreads = 512;  // eight waves, two per SIMD
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

constexpr int NW = 8;                        // waves per workgroup
constexpr int LOADS = TILE_BYTES / 1024 / NW;  // 1 KB direct loads per wave per operand per stage

// One wave's share of a tile: the K loop and the epilogue for MB 32-row A
// blocks from tile row am0 times JW 32-column W blocks from block bw0.  Every
// wave also issues its share of the tile loads: LOADS of the A tile and LW of
// the W tile per stage (LW < LOADS leaves W tile rows past the tile unloaded).
template <int EPI, int MB, int JW, int LW>
__device__ __forceinline__ void gemm_wave(const Params& p, uint8_t* smem, const uint16_t* const (&asrc)[LOADS],
                                          const uint16_t* const (&wsrc)[LOADS], int nk, int wave, int lane,
                                          int m0, int n0, int am0, int bw0, int ks) {
  constexpr int SLOTS = MB * JW;  // MFMAs per 16-wide K slice
  constexpr int RD = MB + JW;     // fragment reads per slice
  constexpr int LA = LOADS;       // A loads per stage
  constexpr int NL = LA + LW;     // direct loads per slice that carries them
  static_assert(RD <= SLOTS && LW <= LOADS, "a slice's slots issue its reads");

  // Step kt's stages; past the last step a load fetches step nk-1 again (into
  // the stage of the step it stands in for, which is never read).
  auto abuf = [&](int kt) { return smem + (kt % SA) * TILE_BYTES; };
  auto wbuf = [&](int kt) { return smem + (SA + kt % SW) * TILE_BYTES; };
  auto src_step = [&](int kt) { return (int64_t)(kt < nk ? kt : nk - 1) * BK; };
  // (named operands: the host pass drops the kernel's launch stub when the
  // builtin's pointer argument is a call expression)
  auto load_one = [&](bool w, int j, int kt) {
    const uint16_t* src = (w ? wsrc[j] : asrc[j]) + src_step(kt);
    uint8_t* dst = (w ? wbuf(kt) : abuf(kt)) + 1024 * (NW * j + wave);
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)dst, 16, 0, 0);
  };

  f32x16 acc[MB][JW];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < JW; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // The K loop is scheduled by hand: each slice is SLOTS MFMA slots; the
  // first slots also issue the fragment reads for the next slice (and, in the
  // slice after the barrier, the direct loads, spread over the slots).
  const int rl = lane & 31, kh = lane >> 5;
  // fragment read q (0..RD-1) of slice s (16 values of K) of step k: weight
  // block q for q < JW, then A block q-JW
  auto read_frag = [&](int k, int s, int q, v4u (&fa)[MB], v4u (&fw)[JW]) {
    const bool w = q < JW;
    const uint8_t* buf = w ? wbuf(k) : abuf(k);
    const int r = w ? 32 * (bw0 + q) + rl : am0 + 32 * (q - JW) + rl;
    const v4u v = *reinterpret_cast<const v4u*>(buf + r * ROW_BYTES + swz(r, 2 * s + kh) * 16);
    if (w) fw[q] = v;
    else fa[q - JW] = v;
  };
  // One slice: the SLOTS MFMAs on (fa, fw), the reads of the next fragments
  // (slice rs of step rk) into (na, nw), RPS per slot from slot 0, and
  // optionally the loads of steps ka (A, issued first) and kw (W).
  auto half = [&](const v4u (&fa)[MB], const v4u (&fw)[JW], int rk, int rs, v4u (&na)[MB], v4u (&nw)[JW],
                  bool load, int ka, int kw) {
    constexpr int RPS = KF_GEMM_READS_PER_SLOT;
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) {
      acc[q / JW][q % JW] = mfma32(fa[q / JW], fw[q % JW], acc[q / JW][q % JW]);
#pragma unroll
      for (int r = 0; r < RPS; ++r)
        if (q * RPS + r < RD) read_frag(rk, rs, q * RPS + r, na, nw);
      if (load) {
#pragma unroll
        for (int l = q * NL / SLOTS; l < (q + 1) * NL / SLOTS; ++l) load_one(l >= LA, l >= LA ? l - LA : l, l >= LA ? kw : ka);
      }
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
    if (s < SA) {
#pragma unroll
      for (int j = 0; j < LA; ++j) load_one(false, j, s);
    }
#pragma unroll
    for (int j = 0; j < LW; ++j) load_one(true, j, s);
  }
  wait_vm<(SA - 1) * LA + (SW - 1) * LW>();  // step 0 has landed
  block_barrier();
  v4u fa[2][MB], fw[2][JW];
#pragma unroll
  for (int q = 0; q < RD; ++q) read_frag(0, 0, q, fa[0], fw[0]);
  static_assert(SS % 2 == 0, "a step starts with its fragments in buffer 0");
  for (int k = 0; k + 1 < nk; ++k) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s + 1 < SS; ++s)
      half(fa[s & 1], fw[s & 1], k, s + 1, fa[(s + 1) & 1], fw[(s + 1) & 1], false, 0, 0);
    // This wave's loads for step k+1 are complete once only later steps' remain
    // in flight: the A loads of steps k+2 .. k+SA-1 and the W loads of steps
    // k+2 .. k+SW-1, which are the most recent ones (A before W within a step).
    wait_vm<(SA - 2) * (LA + LW) + (SW - SA) * LW>();
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

  // Epilogue.  Lane l holds column l % 32 of each block.
  const int rq = 4 * (lane >> 5);
  if (EPI == kGemmSwiGLU) {
    // Each 32-column block holds 16 outputs: columns 0-15 their gate rows,
    // 16-31 their up rows.  Lanes c and c ^ 16 exchange values; the gate lane
    // writes elements v = 0..7 of the pair, the up lane v = 8..15.
    bool bad = false;
    const bool gl = (lane & 16) == 0;
    const int nout = p.N >> 1;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < JW; ++j) {
        float pr[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) pr[v] = __shfl_xor(acc[i][j][v], 16);
        const int col = (n0 >> 1) + 16 * (bw0 + j) + (lane & 15);
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int vv = gl ? v : v + 8;
          const float g = gl ? acc[i][j][v] : pr[v + 8], u = gl ? pr[v] : acc[i][j][v + 8];
          const int row = m0 + am0 + 32 * i + 8 * (vv >> 2) + rq + (vv & 3);
          if (row < p.M && col < nout) p.Cb[(int64_t)row * nout + col] = f16_checked(g / (1.0f + expf(-g)) * u, bad);
        }
      }
    raise_err(p.err_flag, bad, kErrF16Range);
  } else {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + am0 + 32 * i + 8 * (v >> 2) + rq + (v & 3);
        if (row >= p.M) continue;
#pragma unroll
        for (int j = 0; j < JW; ++j) {
          const int col = n0 + 32 * (bw0 + j) + rl;
          if (col >= p.N) continue;
          float* c = p.C + (int64_t)row * p.N + col;
          if (EPI == kGemmResidF32) *c += acc[i][j][v];
          else c[(int64_t)ks * p.M * p.N] = acc[i][j][v];
        }
      }
  }
}

// Tiles of 256 rows x 32 NB columns (NB = 8; 7, 5 or 4 where narrower tiles
// fill the chip in fewer tile-times: see gemm_tile_blocks).  With NB = 8 the
// eight waves are 2 x 4 of 128 x 64; with NB = 7 (5) they are 4 x 2 of 64 x 128
// (96) and 64 x 96 (64), so that with waves dealt to the SIMDs round-robin each
// SIMD holds one of each; with NB = 4, 4 x 2 of 64 x 64.  The W tile is loaded
// as 256 rows for NB = 8 and 7 (rows past 32 NB repeat the tile's last row and
// are not used); for NB = 5 and 4 only the loads that hold the tile's rows are
// issued.
template <int EPI, int NB>
__global__ __launch_bounds__(kGemmThreads) void gemm256_kernel(const Params p) {
  static_assert(NB == 8 || NB == 7 || NB == 5 || NB == 4, "tile widths");
  // SA A tiles, then SW W tiles, each [256 rows][CH swizzled 16-byte chunks]; both fp16.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[(SA + SW) * TILE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  constexpr int TN = 32 * NB;  // tile columns
  const int mt = (p.M + BM - 1) / BM, nt = (p.N + TN - 1) / TN, ntiles = mt * nt;
  const int nwg = ntiles * p.splitk;
  // Tiles sharing a weight panel (same column tile) go to the same XCD, where
  // they reuse it through that XCD's L2 (workgroups are dealt round-robin).
  int bid = blockIdx.x;
  if (nwg % 8 == 0) bid = (bid % 8) * (nwg / 8) + bid / 8;
  const int ks = bid % p.splitk, t = bid / p.splitk;
  const int tm = t % mt, tn = t / mt;
  const int m0 = tm * BM, n0 = tn * TN;
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
    const int rt = r < TN ? r : TN - 1;  // W tile rows past the tile's columns repeat its last row
    // weight tile row rt: for SwiGLU, each 32-row block holds the gate rows
    // (first 16) and the up rows (last 16) of 16 outputs
    int wr;
    const uint16_t* wb;
    if (EPI == kGemmSwiGLU) {
      wr = (n0 >> 1) + 16 * (rt >> 5) + (rt & 15);
      wb = (rt & 16) ? p.W2 : p.W;
    } else {
      wr = n0 + rt;
      wb = p.W;
    }
    if (wr >= w_rows) wr = w_rows - 1;  // columns past N load a valid row; they are never stored
    wsrc[j] = wb + (int64_t)wr * K + (int64_t)k_begin * BK + c * 8;
  }
  if (NB == 8) {
    gemm_wave<EPI, 4, 2, LOADS>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, 128 * (wave / 4), 2 * (wave % 4), ks);
  } else if (NB == 5) {
    // W tile load j of wave w fills rows 8 (8 j + w) ..: rows 0..127 take
    // loads 0 and 1 of every wave, rows 128..159 load 2 of waves 0..3
    static_assert(LOADS == 4, "1 KB loads of 8 rows");
    if (wave < 4) gemm_wave<EPI, 2, 3, 3>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, 64 * wave, 0, ks);
    else gemm_wave<EPI, 2, 2, 2>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, 64 * (wave - 4), 3, ks);
  } else if (NB == 4) {
    gemm_wave<EPI, 2, 2, 2>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, 64 * (wave & 3), 2 * (wave >> 2), ks);
  } else {
#ifndef KF_GEMM_NB7_PAIRS
#define KF_GEMM_NB7_PAIRS 0
#endif
    // 4-block waves and 3-block waves: 0..3 and 4..7, or even and odd
    const bool wide = KF_GEMM_NB7_PAIRS ? (wave & 1) == 0 : wave < 4;
    const int am0 = 64 * (KF_GEMM_NB7_PAIRS ? wave >> 1 : wave & 3);
    // W tile load j of wave w fills rows 8 (8 j + w) ..: the last load of waves
    // 4..7 covers rows 224..255, past the tile, and is left out.
    static_assert(KF_GEMM_NB7_PAIRS || LOADS == 4, "waves 4..7 hold the rows past a 224-column tile");
    if (wide) gemm_wave<EPI, 2, 4, LOADS>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, am0, 0, ks);
    else gemm_wave<EPI, 2, 3, KF_GEMM_NB7_PAIRS ? LOADS : LOADS - 1>(p, smem, asrc, wsrc, nk, wave, lane, m0, n0, am0, 4, ks);
  }
}

}  // namespace

#ifndef KF_GEMM_MAX_SPLIT
#define KF_GEMM_MAX_SPLIT 8  // upper bound on K slices per output tile
#endif

// K slices for tiles of 32 nb columns.
static int splitk_for(int M, int N, int K, int nb) {
  const int tiles = ((M + BM - 1) / BM) * ((N + 32 * nb - 1) / (32 * nb));
  const int k32 = K / 32;
  if (tiles >= 192 || k32 < 128) return 1;  // enough tiles, or a short (cheap) reduction
  int s = KF_GEMM_SPLIT_FLOOR ? 256 / tiles : (256 + tiles - 1) / tiles;
  if (s > k32 / 64) s = k32 / 64;  // keep at least 2048 of K per slice
  if (s > KF_GEMM_MAX_SPLIT) s = KF_GEMM_MAX_SPLIT;
  return s < 1 ? 1 : s;
}

#ifndef KF_GEMM_NARROW
#define KF_GEMM_NARROW 1  // split-K tiles of 160 or 128 columns where they take fewer tile-times
#endif
#ifndef KF_GEMM_NARROW_COST
#define KF_GEMM_NARROW_COST 13  // cost of a narrow tile's column-step, in tenths of a 256-column tile's
#endif
// Tile width of the split-K (partial-sum) launch: the number of 32-column
// blocks (8, 5 or 4) whose grid, tiles x K slices, takes the fewest
// tile-times over the 256 CUs.  A tile-time is its columns times its K steps,
// weighted 1.3x for the narrow tiles: per column-step they measured 1.12-1.34x
// the 256-column tile's (fewer MFMAs per fragment read, and a fuller chip runs
// at a lower clock).  The Qwen3-32B-shaped QKV and output projections (160 of
// the 256 CUs busy with 256-column tiles) gain: 69.4 -> 59.4 and 57.9 -> 48.5 us
// with 160-column tiles, where the unweighted rule's 160-column tiles for its
// down projection (240 workgroups either way) lost 122 -> 140 us and for the
// 70B-shaped QKV projection 83.6 -> 87.3 us.
static int partial_tile_blocks(int M, int N, int K) {
  if (!KF_GEMM_NARROW) return 8;
  const int mt = (M + BM - 1) / BM, nk = K / BK;
  int best = 8;
  int64_t best_cost = 0;
  for (int nb : {8, 5, 4}) {
    const int s = splitk_for(M, N, K, nb);
    const int64_t wgs = (int64_t)mt * ((N + 32 * nb - 1) / (32 * nb)) * s;
    const int64_t cost = (wgs + 255) / 256 * nb * ((nk + s - 1) / s) * (nb == 8 ? 10 : KF_GEMM_NARROW_COST);
    if (nb == 8 || cost < best_cost) {
      best = nb;
      best_cost = cost;
    }
  }
  return best;
}

int gemm_splitk(int M, int N, int K) { return splitk_for(M, N, K, partial_tile_blocks(M, N, K)); }

// 32-column blocks per tile: for the split-K launch see partial_tile_blocks;
// 7 for the SwiGLU launch when 224-column tiles take fewer tile-times than
// 256-column ones over whole rounds of the 256 CUs (70B gate/up: 512 tiles of 7
// blocks in 2 rounds against 448 of 8, the second round three quarters full);
// else 8.
int gemm_tile_blocks(int epi, int M, int N, int K) {
  if (epi == kGemmPartialF32) return partial_tile_blocks(M, N, K);
  if (epi != kGemmSwiGLU) return 8;
  const int mt = (M + BM - 1) / BM;
  auto cost = [&](int nb) { return ((mt * ((N + 32 * nb - 1) / (32 * nb)) + 255) / 256) * nb; };
  return cost(7) < cost(8) ? 7 : 8;
}

hipError_t launch_gemm(int epi, const uint16_t* A, const uint16_t* W, const uint16_t* W2, int M, int N, int K,
                       float* C, uint16_t* Cb, int* err_flag, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0 || K % BK) return hipErrorInvalidValue;
  if (epi == kGemmSwiGLU && N % 32) return hipErrorInvalidValue;  // whole 16-output gate/up blocks
  // the nonlinearity and the residual update need complete sums: only the partial epilogue splits K
  Params p{A, W, W2, M, N, K, epi == kGemmPartialF32 ? gemm_splitk(M, N, K) : 1, C, Cb, err_flag};
  const int nb = gemm_tile_blocks(epi, M, N, K);
  const int grid = ((M + BM - 1) / BM) * ((N + 32 * nb - 1) / (32 * nb)) * p.splitk;
  switch (epi) {
    case kGemmResidF32:
      hipLaunchKernelGGL((gemm256_kernel<kGemmResidF32, 8>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      break;
    case kGemmSwiGLU:
      if (nb == 7) hipLaunchKernelGGL((gemm256_kernel<kGemmSwiGLU, 7>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      else hipLaunchKernelGGL((gemm256_kernel<kGemmSwiGLU, 8>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      break;
    case kGemmPartialF32:
      if (nb == 5) hipLaunchKernelGGL((gemm256_kernel<kGemmPartialF32, 5>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      else if (nb == 4) hipLaunchKernelGGL((gemm256_kernel<kGemmPartialF32, 4>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      else hipLaunchKernelGGL((gemm256_kernel<kGemmPartialF32, 8>), dim3(grid), dim3(kGemmThreads), 0, s, p);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kf

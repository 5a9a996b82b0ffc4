// GEMM kernels: C[m, n] = (R ? R[m, n] : 0) + alpha * sum_k A(m, k) B(n, k).
//
// bf16: gfx950 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation.  Workgroup
// tile 128x128, K step 64, four waves each owning a 64x64 quarter (2x2 MFMA
// blocks).  Both operands are staged in LDS as [row][k] with k contiguous so
// every MFMA fragment is one 16-byte LDS read.  An operand whose k is not
// contiguous in HBM (input and weight gradients) is transposed on its way into
// LDS: each thread loads four k-rows of eight consecutive m/n values (16-byte
// coalesced loads) and writes eight 8-byte [m][k0..k0+3] pieces.  LDS is
// double buffered and the next tile's global loads are issued before the
// current tile's MFMAs, one barrier per K step.
//
// The row count (forward and input-gradient GEMMs) or the reduction length
// (weight-gradient GEMMs) can be read from a device kept count, so the grid is
// sized for the whole batch and tiles past the kept rows exit at once.
//
// fp32: a plain SIMT kernel (64x64 tiles, 4x4 per thread) used by the fp32
// configuration only.
#include <algorithm>
#include <functional>
#include <initializer_list>
#include <queue>
#include <utility>
#include <type_traits>
#include <vector>

#include "ld_internal.h"

namespace ld {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64, LDK = BK + 8;  // LDS row pitch (bf16)
constexpr int kTileElems = BM * LDK;

__device__ __forceinline__ int64_t map_row(const RowMap& m, int64_t row) {
  if (!m.idx) return row;
  return static_cast<int64_t>(m.idx[row / m.S]) * m.S + row % m.S;
}

__device__ __forceinline__ void resolve_counts(const GemmArgs& g, int& M, int& K) {
  M = g.M;
  K = g.K;
  if (g.dev_count) {
    const int c = *g.dev_count * g.count_mult;
    if (g.count_dim == 0)
      M = c;
    else
      K = c;
  }
}

// ---- operand staging -------------------------------------------------------

// k-contiguous operand X[r * ld + k]: 128 rows x 64 k = 1024 chunks of 8.
struct KRegs {
  uint4 v[4];
};
__device__ __forceinline__ void load_kc(KRegs& t, const bf16* X, int64_t ld, int r0, int R, int k0,
                                        int K, int tid) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int chunk = p * 256 + tid;
    const int row = chunk >> 3, kc = (chunk & 7) * 8;
    const int gr = r0 + row, gk = k0 + kc;
    if (gr < R && gk < K)
      t.v[p] = *reinterpret_cast<const uint4*>(X + static_cast<int64_t>(gr) * ld + gk);
    else
      t.v[p] = make_uint4(0, 0, 0, 0);
  }
}
__device__ __forceinline__ void store_kc(const KRegs& t, bf16* lds, int tid) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int chunk = p * 256 + tid;
    const int row = chunk >> 3, kc = (chunk & 7) * 8;
    *reinterpret_cast<uint4*>(lds + row * LDK + kc) = t.v[p];
  }
}

// mn-contiguous operand X[k * ld + r]: thread loads k-rows kg..kg+3 of the
// eight r values rc..rc+7 and writes them transposed.
__device__ __forceinline__ void load_mc(KRegs& t, const bf16* X, int64_t ld, int r0, int R, int k0,
                                        int K, int tid) {
  const int rc = (tid & 15) * 8, kg = (tid >> 4) * 4;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int gk = k0 + kg + kk, gr = r0 + rc;
    if (gk < K && gr < R)
      t.v[kk] = *reinterpret_cast<const uint4*>(X + static_cast<int64_t>(gk) * ld + gr);
    else
      t.v[kk] = make_uint4(0, 0, 0, 0);
  }
}
__device__ __forceinline__ uint32_t half_of(const uint4& v, int i) {
  const uint32_t w = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
  return (i & 1) ? (w >> 16) : (w & 0xffffu);
}
__device__ __forceinline__ void store_mc(const KRegs& t, bf16* lds, int tid) {
  const int rc = (tid & 15) * 8, kg = (tid >> 4) * 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint2 o;
    o.x = half_of(t.v[0], i) | (half_of(t.v[1], i) << 16);
    o.y = half_of(t.v[2], i) | (half_of(t.v[3], i) << 16);
    *reinterpret_cast<uint2*>(lds + (rc + i) * LDK + kg) = o;
  }
}

template <bool KC>
__device__ __forceinline__ void load_op(KRegs& t, const bf16* X, int64_t ld, int r0, int R, int k0,
                                        int K, int tid) {
  if constexpr (KC)
    load_kc(t, X, ld, r0, R, k0, K, tid);
  else
    load_mc(t, X, ld, r0, R, k0, K, tid);
}
template <bool KC>
__device__ __forceinline__ void store_op(const KRegs& t, bf16* lds, int tid) {
  if constexpr (KC)
    store_kc(t, lds, tid);
  else
    store_mc(t, lds, tid);
}

// ---- epilogue -------------------------------------------------------------
// 32x32 accumulator layout: lane l, register v holds row
// 8*(v/4) + 4*(l/32) + v%4 and column l%32 of the block.
__device__ __forceinline__ void epilogue_store(const GemmArgs& g, float alpha, int row, int col,
                                               float acc, int M) {
  if (row >= M || col >= g.N) return;
  float val = alpha * acc;
  const int64_t orow = map_row(g.out_map, row);
  if (g.R) {
    const int64_t rrow = g.r_mapped ? orow : row;
    if (g.r_f32)
      val += static_cast<const float*>(g.R)[rrow * g.ldr + col];
    else
      val += static_cast<float>(static_cast<const bf16*>(g.R)[rrow * g.ldr + col]);
  }
  if (g.c_f32)
    static_cast<float*>(g.C)[orow * g.ldc + col] = val;
  else
    static_cast<bf16*>(g.C)[orow * g.ldc + col] = static_cast<bf16>(val);
}

template <bool AK, bool BKC>
__device__ __forceinline__ void gemm_bf16_body(const GemmArgs& g) {
  extern __shared__ __align__(16) bf16 smem[];
  bf16* As = smem;                  // [2][BM][LDK]
  bf16* Bs = smem + 2 * kTileElems;  // [2][BN][LDK]
  int M, K;
  resolve_counts(g, M, K);
  const int tiles_n = (g.N + BN - 1) / BN;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  if (m0 >= M) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* B = static_cast<const bf16*>(g.B);

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = (K + BK - 1) / BK;
  if (nk > 0) {
    KRegs ra, rb;
    load_op<AK>(ra, A, g.lda, m0, M, 0, K, tid);
    load_op<BKC>(rb, B, g.ldb, n0, g.N, 0, K, tid);
    store_op<AK>(ra, As, tid);
    store_op<BKC>(rb, Bs, tid);
    __syncthreads();
    const int lrow = lane & 31, lk = (lane >> 5) * 8;
    for (int kt = 0; kt < nk; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nk) {
        load_op<AK>(ra, A, g.lda, m0, M, (kt + 1) * BK, K, tid);
        load_op<BKC>(rb, B, g.ldb, n0, g.N, (kt + 1) * BK, K, tid);
      }
      const bf16* as = As + buf * kTileElems;
      const bf16* bs = Bs + buf * kTileElems;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8 af[2], bfr[2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          af[i] = *reinterpret_cast<const bf16x8*>(as + (wm * 64 + i * 32 + lrow) * LDK + ks * 16 + lk);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bfr[j] = *reinterpret_cast<const bf16x8*>(bs + (wn * 64 + j * 32 + lrow) * LDK + ks * 16 + lk);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
      if (kt + 1 < nk) {
        store_op<AK>(ra, As + (buf ^ 1) * kTileElems, tid);
        store_op<BKC>(rb, Bs + (buf ^ 1) * kTileElems, tid);
      }
      __syncthreads();
    }
  }
  const float alpha = g.alpha * (g.alpha_dev ? *g.alpha_dev : 1.f);
  const int half = lane >> 5, col_l = lane & 31;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
        const int col = n0 + wn * 64 + j * 32 + col_l;
        epilogue_store(g, alpha, row, col, acc[i][j][v], M);
      }
}

__global__ __launch_bounds__(256) void ld_gemm_bf16_nt(GemmArgs g) { gemm_bf16_body<true, true>(g); }
__global__ __launch_bounds__(256) void ld_gemm_bf16_nn(GemmArgs g) { gemm_bf16_body<true, false>(g); }
__global__ __launch_bounds__(256) void ld_gemm_bf16_tn(GemmArgs g) { gemm_bf16_body<false, false>(g); }
__global__ __launch_bounds__(256) void ld_gemm_bf16_tt(GemmArgs g) { gemm_bf16_body<false, true>(g); }

// ---- fp32 SIMT ------------------------------------------------------------

constexpr int FT = 64, FK = 16;

template <bool AK, bool BKC>
__global__ __launch_bounds__(256) void ld_gemm_f32_k(GemmArgs g) {
  __shared__ float As[FK][FT + 4], Bs[FK][FT + 4];
  int M, K;
  resolve_counts(g, M, K);
  const int tiles_n = (g.N + FT - 1) / FT;
  const int m0 = (blockIdx.x / tiles_n) * FT, n0 = (blockIdx.x % tiles_n) * FT;
  if (m0 >= M) return;
  const float* A = static_cast<const float*>(g.A);
  const float* B = static_cast<const float*>(g.B);
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int id = e * 256 + tid;
      int mm, kk;
      if (AK) { mm = id / FK; kk = id % FK; } else { kk = id / FT; mm = id % FT; }
      const int gm = m0 + mm, gk = k0 + kk;
      float v = 0.f;
      if (gm < M && gk < K) v = AK ? A[static_cast<int64_t>(gm) * g.lda + gk] : A[static_cast<int64_t>(gk) * g.lda + gm];
      As[kk][mm] = v;
      int nn;
      if (BKC) { nn = id / FK; kk = id % FK; } else { kk = id / FT; nn = id % FT; }
      const int gn = n0 + nn, gk2 = k0 + kk;
      float w = 0.f;
      if (gn < g.N && gk2 < K) w = BKC ? B[static_cast<int64_t>(gn) * g.ldb + gk2] : B[static_cast<int64_t>(gk2) * g.ldb + gn];
      Bs[kk][nn] = w;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[kk][ty * 4 + r];
#pragma unroll
      for (int c = 0; c < 4; ++c) b[c] = Bs[kk][tx * 4 + c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = __builtin_fmaf(a[r], b[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int row = m0 + ty * 4 + r, col = n0 + tx * 4 + c;
      if (row >= M || col >= g.N) continue;
      float val = g.alpha * (g.alpha_dev ? *g.alpha_dev : 1.f) * acc[r][c];
      const int64_t orow = map_row(g.out_map, row);
      if (g.R) val += static_cast<const float*>(g.R)[(g.r_mapped ? orow : row) * g.ldr + col];
      static_cast<float*>(g.C)[orow * g.ldc + col] = val;
    }
}

constexpr size_t kGemmLds = 4 * kTileElems * sizeof(bf16);

// ===================================================================== big
// 256x256 workgroup tile, four waves in a 2x2 grid each owning 128x128 (4x4
// MFMA blocks, 256 fp32 accumulators per lane), k walked in tiles of 32.
//
// Operand tiles go from global memory straight into LDS: buffer loads with an
// LDS destination, so no register staging and no LDS write instructions.
// Such a load writes the 16 bytes of lane i at LDS offset 16*i from a
// wave-uniform base, so the LDS layout is set by which global chunk each lane
// fetches.  Each operand has a region of the ring:
//   mn-contiguous operand: four stages of one k tile, [32 k][256 mn] as in
//     memory, chunks XOR-swizzled by k; a load instruction fetches two whole
//     512-byte k rows.  A fragment is two transposing reads
//     (ds_read_b64_tr_b16: in each group of 16 lanes, lane j receives element
//     j%4 of the four-element rows read by lanes j/4, j/4+4, j/4+8 and
//     j/4+12, so 16 lanes reading rows k..k+3 at mn offsets 0, 4, 8, 12 give
//     lane j the values k..k+3 at mn j).
//   k-contiguous operand: slots of a PAIR of k tiles, [256 rows][64 k], so
//     a load instruction fetches 8 rows as whole 128-byte lines (a single k
//     tile is 64 bytes of a row: half lines, twice the cache requests for
//     the same bytes).  Two slots, or three for A when both operands are
//     k-contiguous (96 KB; the ring is then the whole 160 KB of LDS).  The
//     16-byte chunks of a row are XOR-swizzled by the row; a fragment is one
//     16-byte read per lane.
// Rows past the operand's end, and k chunks past the split's end, are
// fetched from an offset outside the buffer descriptor's range and land in
// LDS as zeros.  The loads are issued as inline assembly (ld_internal.h),
// so the compiler does not track them; the kernel waits for them itself
// (s_waitcnt vmcnt) before the barriers.
//
// Per k tile (two k-substeps of 16): one barrier at the top, where each wave
// has waited until the next tile has landed; then the tile's 32 MFMAs run on
// fragments read during the previous tile, next to the reads of all of the
// next tile's fragments and the loads for later tiles: an mn-contiguous
// stage is reloaded (tile kt+4) during the tile kt it holds, whose fragments
// were read before the barrier; a k-contiguous slot is reloaded once both
// of its tiles have been read: with two slots, pair kt+3, kt+4 during odd
// tiles kt; A's third slot lets its pair kt+5, kt+6 load half during odd
// tile kt and half during kt+1.  Every load has at least one tile-time,
// most two or more, to land.  No MFMA waits on a recent LDS read.
//
// The MFMA is issued as B x A so each lane ends with 4 consecutive output
// columns of one row.  Tiles are ordered XCD-aware: consecutive workgroup ids
// go to different XCDs, so ids are remapped to give each XCD a contiguous
// range of tiles, walked in groups of 8 tile-rows for L2 reuse.  Split-K
// (grid.y) writes fp32 partials that a second kernel sums in split order.

constexpr int GB = 256, GK = 32;
constexpr int kBigTile = GB * GK;       // elements of one operand's k tile
constexpr int kLoadsMC = 4;             // load instructions per wave per mn-contiguous tile
constexpr int kLoadsKC = 8;             // load instructions per wave per k-contiguous pair
constexpr int kStagePitch = 132;        // floats per staged epilogue row (128 + 4 pad)
constexpr int kStagePitch16 = 132;      // bf16 per staged row of a bf16 epilogue (264 bytes)
constexpr uint32_t kOob = kDmaOob;
constexpr int64_t kBigMaxSpan = kDmaMaxSpan;
// Ring regions (elements): a k-contiguous A takes three pair slots when B
// is k-contiguous too, every other operand four tile stages or two pair
// slots (64 KB).
template <bool AK, bool BKC>
constexpr int slots_a() { return AK && BKC ? 3 : 2; }
template <bool AK, bool BKC>
constexpr int region_a() { return AK ? slots_a<AK, BKC>() * 2 * kBigTile : 4 * kBigTile; }
template <bool AK, bool BKC>
constexpr int ring_elems() { return region_a<AK, BKC>() + 4 * kBigTile; }
static_assert(ring_elems<true, true>() * 2 <= 160 * 1024, "the ring fits the LDS");
static_assert(ring_elems<false, false>() * 2 >= 4 * 32 * kStagePitch * 4, "epilogue staging fits the ring");

typedef short v4s __attribute__((ext_vector_type(4)));
typedef dma_rsrc v4i;
#define LD_LDS(T, p) ((__attribute__((address_space(3))) T*)(p))

// Element offset, in an operand's region, of the stage (mn-contiguous) or
// pair slot (k-contiguous, NS slots) holding k tile kt.
template <bool KC, int NS>
__device__ __forceinline__ int tile_base(int kt) {
  if constexpr (KC)
    return ((kt >> 1) % NS) * (2 * kBigTile);
  else
    return (kt & 3) * kBigTile;
}

// k-contiguous pair slot: element (row, k) of a [256][64] slot.  The chunk
// swizzle uses row bits 1-3: of 16 lanes reading one chunk of 16
// consecutive rows, the two rows of each pair sit 128 bytes apart and the 8
// pairs on 8 different chunks, so all 16 hit different 16-byte bank groups;
// moving by a multiple of 16 rows is a plain offset.
__device__ __forceinline__ int kc_swz(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swz_off(int row, int k) {
  return row * (2 * GK) + ((((k >> 3) ^ kc_swz(row)) << 3) | (k & 7));
}

// mn-contiguous tile: element (k, m) of a [32][256] tile.  The swizzle puts
// the 4 k rows a 16-lane transposing read touches (32 bytes each) on 4
// different 64-byte bank groups, and rows k and k+8 on different halves; it
// depends on k bits 0, 1 and 3 only, so k steps of 4 and 16 are plain offsets.
__device__ __forceinline__ int mc_swz(int k) { return ((k & 3) << 2) | (((k >> 3) & 1) << 1); }
__device__ __forceinline__ int mc_off(int k, int m) {
  return k * GB + ((((m >> 3) ^ mc_swz(k)) << 3) | (m & 7));
}

// Per-lane constants of one operand's tile loads and fragment reads.
template <bool KC>
struct OpLanes {
  uint32_t ld_off[2];  // byte offset of the lane's first 16-byte chunk (mn: per k-row parity)
  int kchunk;          // k-contiguous: k offset of the lane's chunk in the pair
  int frag[4];         // element offsets of fragment reads: per (k half, k-substep) (KC) or block (MC)
};

// `r`: the first of the wave's 128 fragment rows (0 or 128).
template <bool KC>
__device__ __forceinline__ OpLanes<KC> op_lanes(int64_t ld, int lane, int wave, int r) {
  OpLanes<KC> o;
  if constexpr (KC) {
    // load instruction p fills slot rows 8 (4p + wave) .. +7, lane -> row
    // + lane/8, physical chunk lane%8; the swizzle is the same for every p
    const int row = wave * 8 + (lane >> 3);
    o.kchunk = ((lane & 7) ^ kc_swz(row)) << 3;
    o.ld_off[0] = o.ld_off[1] = static_cast<uint32_t>((static_cast<int64_t>(row) * ld + o.kchunk) * 2);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        o.frag[2 * h + ks] = swz_off(r + (lane & 31), h * GK + ks * 16 + (lane >> 5) * 8);
  } else {
    // load instruction p fills k rows 8p + 2*wave + lane/32, physical chunk
    // lane%32; the swizzle depends on p only through its parity (k bit 3)
    const int kr = 2 * wave + (lane >> 5);
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int m = ((lane & 31) ^ mc_swz(8 * par + kr)) << 3;
      o.ld_off[par] = static_cast<uint32_t>((static_cast<int64_t>(kr) * ld + m) * 2);
    }
    o.kchunk = 0;
    // transposing reads: lane reads k row kl, 4 elements from mn ml
    const int kl = (lane >> 5) * 8 + ((lane >> 2) & 3);
    const int ml = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
#pragma unroll
    for (int i = 0; i < 4; ++i) o.frag[i] = mc_off(kl, r + ml + 32 * i);
  }
  return o;
}

// Load instruction p of operand X's rows r0.. into `lds` (its stage or
// slot), 16 bytes per lane.  mn-contiguous: instruction p (0-3) fills 2 k
// rows per wave of the tile at k0.  k-contiguous: instruction p (0-7) fills
// 8 rows per wave of the pair at k0 (64 k).  Columns past the end of a valid
// row read real memory; they only reach outputs that are never stored,
// except a k tail of a k-contiguous operand, which is fetched out of range
// (zeros), as is everything of a tile that starts at or past K.
template <bool KC>
__device__ __forceinline__ void tile_part(bf16* lds, const OpLanes<KC>& o, const bf16* X, int64_t ld,
                                          int r0, int R, int k0, int K, int wave, int p) {
  if constexpr (KC) {
    const v4i rs = dma_make_rsrc(X + static_cast<int64_t>(r0) * ld, (static_cast<int64_t>(R) - r0) * ld * 2);
    const uint32_t u = static_cast<uint32_t>((static_cast<int64_t>(p) * 32 * ld + k0) * 2);
    const uint32_t off = k0 + o.kchunk < K ? o.ld_off[0] + u : kOob;
    dma16(rs, lds + (p * 4 + wave) * 512, off);
  } else {
    const v4i rs = dma_make_rsrc(X + static_cast<int64_t>(k0) * ld, (static_cast<int64_t>(K) - k0) * ld * 2);
    const uint32_t u = static_cast<uint32_t>((static_cast<int64_t>(p) * 8 * ld + r0) * 2);
    dma16(rs, lds + (p * 4 + wave) * 512, o.ld_off[p & 1] + u);
  }
  (void)R;
}

// B slot of the fused SwiGLU forward: the slot's 64-row block b = p/2 holds
// gate rows (b even) or up rows (b odd) tn*128 + (b/2)*64 .. +63 of
// W_gate_up [2f, K], so the tile holds [gate 0-63 | up 0-63 | gate 64-127 |
// up 64-127] of its 128 d_ff columns and each wave's 128 rows pair every
// gate row with its up row 64 further on.  Instruction p (0-7) fills rows
// 32 (p%2) + 8 wave .. +7 of block b.
__device__ __forceinline__ void tile_part_glu(bf16* lds, const OpLanes<true>& o, const bf16* W, int64_t ld,
                                              int tn, int f, int k0, int K, int wave, int p) {
  const int b = p >> 1;
  const int64_t rbase = ((b & 1) ? f : 0) + static_cast<int64_t>(tn) * 128 + (b >> 1) * 64;
  const v4i rs = dma_make_rsrc(W + rbase * ld, 64 * ld * 2);
  const uint32_t u = static_cast<uint32_t>((static_cast<int64_t>(p & 1) * 32 * ld + k0) * 2);
  const uint32_t off = k0 + o.kchunk < K ? o.ld_off[0] + u : kOob;
  dma16(rs, lds + (p * 4 + wave) * 512, off);
}

// Fragment of block i of the wave's 128 rows for k-substep ks of the tile
// whose stage or slot starts at t (h: the tile's half of a k-contiguous
// pair): the lane's MFMA row is r + 32 i + lane % 32 (r as given to
// op_lanes), its 8 k values start at ks*16 + (lane/32)*8.  Only the per-lane
// offset is a register; the rest is a constant offset of the LDS instruction.
template <bool KC>
__device__ __forceinline__ bf16x8 frag(const bf16* t, const OpLanes<KC>& o, int i, int h, int ks) {
  if constexpr (KC) {
    return *reinterpret_cast<const bf16x8*>(t + 32 * i * (2 * GK) + o.frag[2 * h + ks]);
  } else {
    (void)h;
    const bf16* p = t + o.frag[i] + ks * 16 * GB;
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LD_LDS(v4s, p));
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LD_LDS(v4s, p + 4 * GB));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }
}

// Tile of workgroup `pid` among the n_valid = tiles_m * tiles_n tiles that
// hold rows (tiles_m counts only tile rows below the kept count), or false
// when the workgroup has none.  Workgroup ids are dealt to the 8 XCDs in
// turn (id % 8), so XCD x is given its own contiguous, balanced range of
// n_valid / 8 (+1) tiles: the tiles of rows past the kept count are not
// piled onto the last XCDs, and consecutive tiles share an XCD's L2.  Within
// a range, tiles go in groups of 8 tile rows, column by column.  The grid has
// at least as many ids per XCD as the largest range (it is sized for every
// row), so every tile is taken.
__device__ __forceinline__ bool tile_coords(int pid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int n_valid = tiles_m * tiles_n;
  const int x = pid & 7, li = pid >> 3;
  const int base = n_valid >> 3, rem = n_valid & 7;
  if (li >= base + (x < rem ? 1 : 0)) return false;
  const int t = x * base + min(x, rem) + li;
  constexpr int G = 8;
  const int group = G * tiles_n;
  const int first_m = (t / group) * G;
  const int gsz = min(tiles_m - first_m, G);
  const int in = t % group;
  tm = first_m + in % gsz;
  tn = in / gsz;
  return true;
}

// Epilogue of one staged 32-row block row: the lane's rows are r0 + 2 it
// (it = 0..15), its 4 columns n..n+3; the staged values (alpha applied) sit
// at stage[(2 it + half) * kStagePitch + c].
//
// Full block row (every row < M, every column < N): all staged values, row
// map entries and residual values are requested before the first store, so
// their latencies overlap, and no branch splits the rows.
__device__ __forceinline__ void epilogue_rows_full(const GemmArgs& g, float* part, const float* stage,
                                                   int r0, int half, int c, int n, int q_last) {
  float4 v[16];
#pragma unroll
  for (int it = 0; it < 16; ++it)
    v[it] = *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c);
  if (part) {
#pragma unroll
    for (int it = 0; it < 16; ++it)
      *reinterpret_cast<float4*>(part + static_cast<int64_t>(r0 + 2 * it) * g.N + n) = v[it];
    return;
  }
  int32_t orow[16];
  if (g.out_map.idx) {
    // output row = idx[r / S] * S + r % S
    const int S = g.out_map.S;
    const int q0 = r0 / S, rem0 = r0 - q0 * S;
    if (S >= 32) {
      // the 32 rows span at most two sequences
      const int s0 = g.out_map.idx[q0], s1 = g.out_map.idx[min(q0 + 1, q_last)];
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int rr = rem0 + 2 * it;
        orow[it] = rr >= S ? s1 * S + (rr - S) : s0 * S + rr;
      }
    } else {
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int r = r0 + 2 * it, q = r / S;
        orow[it] = g.out_map.idx[q] * S + (r - q * S);
      }
    }
  } else {
#pragma unroll
    for (int it = 0; it < 16; ++it) orow[it] = r0 + 2 * it;
  }
  if (g.R && g.r_f32) {  // float32 residual (the residual streams)
    const float* R = static_cast<const float*>(g.R);
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // two halves of 8 rows: fewer registers live
      float4 rv[8];
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int64_t rrow = g.r_mapped ? orow[8 * h + it] : r0 + 2 * (8 * h + it);
        rv[it] = *reinterpret_cast<const float4*>(R + rrow * g.ldr + n);
      }
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        float4& t = v[8 * h + it];
        t.x += rv[it].x;
        t.y += rv[it].y;
        t.z += rv[it].z;
        t.w += rv[it].w;
      }
    }
  } else if (g.R) {  // bf16 residual
    uint2 rv[16];
    const bf16* R = static_cast<const bf16*>(g.R);
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int64_t rrow = g.r_mapped ? orow[it] : r0 + 2 * it;
      rv[it] = *reinterpret_cast<const uint2*>(R + rrow * g.ldr + n);
    }
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const bf16* rb = reinterpret_cast<const bf16*>(&rv[it]);
      v[it].x += static_cast<float>(rb[0]);
      v[it].y += static_cast<float>(rb[1]);
      v[it].z += static_cast<float>(rb[2]);
      v[it].w += static_cast<float>(rb[3]);
    }
  }
  if (g.c_f32) {
#pragma unroll
    for (int it = 0; it < 16; ++it)
      *reinterpret_cast<float4*>(static_cast<float*>(g.C) + static_cast<int64_t>(orow[it]) * g.ldc + n) = v[it];
  } else {
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      __attribute__((aligned(8))) bf16 o[4] = {static_cast<bf16>(v[it].x), static_cast<bf16>(v[it].y),
                                               static_cast<bf16>(v[it].z), static_cast<bf16>(v[it].w)};
      *reinterpret_cast<uint2*>(static_cast<bf16*>(g.C) + static_cast<int64_t>(orow[it]) * g.ldc + n) =
          *reinterpret_cast<const uint2*>(o);
    }
  }
}

// Block row with rows past M or columns past N: one row at a time, each
// checked.
__device__ __forceinline__ void epilogue_rows_edge(const GemmArgs& g, float* part, const float* stage,
                                                   int r0, int half, int c, int n, int M) {
#pragma unroll 1
  for (int it = 0; it < 16; ++it) {
    const int m = r0 + 2 * it;
    if (m >= M || n >= g.N) continue;
    float4 v = *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c);
    if (part) {
      *reinterpret_cast<float4*>(part + static_cast<int64_t>(m) * g.N + n) = v;
      continue;
    }
    const int64_t orow = map_row(g.out_map, m);
    if (g.R) {
      const int64_t rrow = g.r_mapped ? orow : m;
      if (g.r_f32) {
        const float4 r = *reinterpret_cast<const float4*>(static_cast<const float*>(g.R) + rrow * g.ldr + n);
        v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
      } else {
        const uint2 r = *reinterpret_cast<const uint2*>(static_cast<const bf16*>(g.R) + rrow * g.ldr + n);
        const bf16* rb = reinterpret_cast<const bf16*>(&r);
        v.x += static_cast<float>(rb[0]); v.y += static_cast<float>(rb[1]);
        v.z += static_cast<float>(rb[2]); v.w += static_cast<float>(rb[3]);
      }
    }
    if (g.c_f32) {
      *reinterpret_cast<float4*>(static_cast<float*>(g.C) + orow * g.ldc + n) = v;
    } else {
      __attribute__((aligned(8))) bf16 o[4] = {static_cast<bf16>(v.x), static_cast<bf16>(v.y),
                                               static_cast<bf16>(v.z), static_cast<bf16>(v.w)};
      *reinterpret_cast<uint2*>(static_cast<bf16*>(g.C) + orow * g.ldc + n) = *reinterpret_cast<const uint2*>(o);
    }
  }
}

constexpr int kEpiPlain = 0, kEpiGluFwd = 1, kEpiGluBwd = 2, kEpiRelu2Fwd = 3, kEpiRelu2Bwd = 4;

__device__ __forceinline__ uint2 pack4_bf16(float a, float b, float c, float d) {
  __attribute__((aligned(8))) bf16 o[4] = {static_cast<bf16>(a), static_cast<bf16>(b), static_cast<bf16>(c),
                                           static_cast<bf16>(d)};
  return *reinterpret_cast<const uint2*>(o);
}

__device__ __forceinline__ float4 unpack4_bf16(uint2 r) {
  const bf16* b = reinterpret_cast<const bf16*>(&r);
  return make_float4(static_cast<float>(b[0]), static_cast<float>(b[1]), static_cast<float>(b[2]),
                     static_cast<float>(b[3]));
}

// Fused SwiGLU backward: the staged gs values (alpha applied; rows r0 + 2 it,
// columns n..n+3 < N = f), kept in float32 (gs is never stored), with u and
// v read from aux, give gu and gv in C columns n and f + n.
__device__ __forceinline__ void glu_bwd_one(const GemmArgs& g, float4 gs, uint2 ur, uint2 vr, int64_t m, int n) {
  const float4 u = unpack4_bf16(ur), v = unpack4_bf16(vr);
  float gu[4], gv[4];
  swiglu_bwd_f(u.x, v.x, gs.x, gu[0], gv[0]);
  swiglu_bwd_f(u.y, v.y, gs.y, gu[1], gv[1]);
  swiglu_bwd_f(u.z, v.z, gs.z, gu[2], gv[2]);
  swiglu_bwd_f(u.w, v.w, gs.w, gu[3], gv[3]);
  bf16* C = static_cast<bf16*>(g.C) + m * g.ldc;
  *reinterpret_cast<uint2*>(C + n) = pack4_bf16(gu[0], gu[1], gu[2], gu[3]);
  *reinterpret_cast<uint2*>(C + g.glu_f + n) = pack4_bf16(gv[0], gv[1], gv[2], gv[3]);
}

__device__ __forceinline__ void glu_bwd_rows(const GemmArgs& g, const float* stage, int r0, int half, int c, int n,
                                             int M, bool full) {
  const bf16* U = static_cast<const bf16*>(g.aux);
  const int64_t ldu = 2ll * g.glu_f;
  if (full) {
    uint2 ur[16], vr[16];
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int64_t m = r0 + 2 * it;
      ur[it] = *reinterpret_cast<const uint2*>(U + m * ldu + n);
      vr[it] = *reinterpret_cast<const uint2*>(U + m * ldu + g.glu_f + n);
    }
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const float4 gs = *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c);
      glu_bwd_one(g, gs, ur[it], vr[it], r0 + 2 * it, n);
    }
  } else {
#pragma unroll 1
    for (int it = 0; it < 16; ++it) {
      const int64_t m = r0 + 2 * it;
      if (m >= M || n >= g.N) continue;
      const float4 gs = *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c);
      glu_bwd_one(g, gs, *reinterpret_cast<const uint2*>(U + m * ldu + n),
                  *reinterpret_cast<const uint2*>(U + m * ldu + g.glu_f + n), m, n);
    }
  }
}

// Fused squared-ReLU forward: staged values (alpha applied) of rows r0 + 2 it,
// columns n..n+3, go to C as u (bf16, kept for the backward) and to aux as
// s = relu(u)^2 of the float32 u (one rounding fewer than from a stored u).
__device__ __forceinline__ void relu2_fwd_one(const GemmArgs& g, float4 v, int64_t m, int n) {
  const float u[4] = {v.x, v.y, v.z, v.w};
  float q[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float z = fmaxf(u[e], 0.f);
    q[e] = z * z;
  }
  *reinterpret_cast<uint2*>(static_cast<bf16*>(g.C) + m * g.ldc + n) = pack4_bf16(u[0], u[1], u[2], u[3]);
  *reinterpret_cast<uint2*>(static_cast<bf16*>(g.aux) + m * g.glu_f + n) = pack4_bf16(q[0], q[1], q[2], q[3]);
}

__device__ __forceinline__ void relu2_fwd_rows(const GemmArgs& g, const float* stage, int r0, int half, int c,
                                               int n, int M, bool full) {
  if (full) {
    float4 v[16];
#pragma unroll
    for (int it = 0; it < 16; ++it) v[it] = *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c);
#pragma unroll
    for (int it = 0; it < 16; ++it) relu2_fwd_one(g, v[it], r0 + 2 * it, n);
  } else {
#pragma unroll 1
    for (int it = 0; it < 16; ++it) {
      const int64_t m = r0 + 2 * it;
      if (m >= M || n >= g.N) continue;
      relu2_fwd_one(g, *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c), m, n);
    }
  }
}

// Fused squared-ReLU backward: the staged gs values, kept in float32 (gs is
// never stored), with u read from aux, give gu = gs 2 relu(u) in C.
__device__ __forceinline__ void relu2_bwd_one(const GemmArgs& g, float4 gs, uint2 ur, int64_t m, int n) {
  const float4 u = unpack4_bf16(ur);
  *reinterpret_cast<uint2*>(static_cast<bf16*>(g.C) + m * g.ldc + n) =
      pack4_bf16(gs.x * 2.f * fmaxf(u.x, 0.f), gs.y * 2.f * fmaxf(u.y, 0.f), gs.z * 2.f * fmaxf(u.z, 0.f),
                 gs.w * 2.f * fmaxf(u.w, 0.f));
}

__device__ __forceinline__ void relu2_bwd_rows(const GemmArgs& g, const float* stage, int r0, int half, int c,
                                               int n, int M, bool full) {
  const bf16* U = static_cast<const bf16*>(g.aux);
  if (full) {
    uint2 ur[16];
#pragma unroll
    for (int it = 0; it < 16; ++it) ur[it] = *reinterpret_cast<const uint2*>(U + static_cast<int64_t>(r0 + 2 * it) * g.glu_f + n);
#pragma unroll
    for (int it = 0; it < 16; ++it)
      relu2_bwd_one(g, *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c), ur[it],
                    r0 + 2 * it, n);
  } else {
#pragma unroll 1
    for (int it = 0; it < 16; ++it) {
      const int64_t m = r0 + 2 * it;
      if (m >= M || n >= g.N) continue;
      relu2_bwd_one(g, *reinterpret_cast<const float4*>(stage + (2 * it + half) * kStagePitch + c),
                    *reinterpret_cast<const uint2*>(U + m * g.glu_f + n), m, n);
    }
  }
}

// One workgroup's tile of a GEMM: `pid` in [0, n_tiles) picks the tile
// (n_tiles covers every row the grid was sized for), `sp` of `splits` the
// k range; `ring` is the workgroup's LDS.
// Plain bf16 output of a 32-row block row that crosses M: straight from the
// accumulators, each row checked (lane: row lm, columns j*32 + 8q + 4 half).
__device__ __forceinline__ void epilogue_plain_edge_bf16(const GemmArgs& g, const floatx16 (&acc)[4], float alpha,
                                                         int mb, int nb, int lm, int half, int M) {
  if (mb + lm >= M) return;
  bf16* C = static_cast<bf16*>(g.C) + static_cast<int64_t>(mb + lm) * g.ldc + nb;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const floatx16& a = acc[j];
      *reinterpret_cast<uint2*>(C + j * 32 + 8 * q + 4 * half) =
          pack4_bf16(alpha * a[4 * q], alpha * a[4 * q + 1], alpha * a[4 * q + 2], alpha * a[4 * q + 3]);
    }
}

template <bool AK, bool BKC, int EPI = kEpiPlain>
__device__ __forceinline__ void gemm_big_body(const GemmArgs& g, bf16* ring, int pid, int n_tiles, int sp,
                                              int splits) {
  int M, K;
  resolve_counts(g, M, K);
  const int tiles_n = (g.N + GB - 1) / GB;
  const int tiles_m = min(n_tiles / tiles_n, (M + GB - 1) / GB);
  int tm, tn;
  if (!tile_coords(pid, tiles_m, tiles_n, tm, tn)) return;
  const int m0 = tm * GB, n0 = tn * GB;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* B = static_cast<const bf16*>(g.B);

  // k range of this split
  const int nkt_all = (K + GK - 1) / GK;
  const int kt0 = static_cast<int>((static_cast<int64_t>(nkt_all) * sp) / splits);
  const int kt1 = static_cast<int>((static_cast<int64_t>(nkt_all) * (sp + 1)) / splits);
  const int nk = kt1 - kt0;
  const int kend = min(K, kt1 * GK);  // loads at or past it read zeros

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const OpLanes<AK> oa = op_lanes<AK>(g.lda, lane, wave, wm * 128);
  const OpLanes<BKC> ob = op_lanes<BKC>(g.ldb, lane, wave, wn * 128);
  constexpr int NSA = slots_a<AK, BKC>(), NSB = 2;  // pair slots of a k-contiguous A, B
  bf16* const ra = ring;                            // A's region
  bf16* const rb = ring + region_a<AK, BKC>();      // B's region
  // Load instruction q of A or B into the stage of tile kt (mn-contiguous,
  // q 0-3) or the slot of the pair starting at tile kt (k-contiguous, q 0-7).
  auto load_a = [&](int kt, int q) {
    tile_part<AK>(ra + tile_base<AK, NSA>(kt), oa, A, g.lda, m0, M, (kt0 + kt) * GK, kend, wave, q);
  };
  auto load_b = [&](int kt, int q) {
    if constexpr (EPI == kEpiGluFwd)
      tile_part_glu(rb + tile_base<true, NSB>(kt), ob, B, g.ldb, tn, g.glu_f, (kt0 + kt) * GK, kend, wave, q);
    else
      tile_part<BKC>(rb + tile_base<BKC, NSB>(kt), ob, B, g.ldb, n0, g.N, (kt0 + kt) * GK, kend, wave, q);
  };
  // The ring starts full: per k tile t = 0..3, A's then B's loads of that
  // tile (a k-contiguous operand loads its pair at even t), then, with three
  // A slots, the first half of A's pair at tiles 4, 5; zeros past the
  // split's end.
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int q = 0; q < (AK ? kLoadsKC : kLoadsMC); ++q)
      if (!AK || t % 2 == 0) load_a(t, q);
#pragma unroll
    for (int q = 0; q < (BKC ? kLoadsKC : kLoadsMC); ++q)
      if (!BKC || t % 2 == 0) load_b(t, q);
  }
  if constexpr (NSA == 3) {
#pragma unroll
    for (int q = 0; q < kLoadsKC / 2; ++q) load_a(4, q);
  }
  // Loads that may still be in flight at the barriers (counted over the issue
  // order of the first fill and of the tiles, below): at the first barrier,
  // and at the top of even and odd tiles.
  constexpr int kWaitFirst = NSA == 3 ? 20 : AK && BKC ? 16 : AK || BKC ? 20 : 24;
  constexpr int kWaitEven = 16;
  constexpr int kWaitOdd = NSA == 3 ? 4 : AK && BKC ? 0 : BKC ? 4 : AK ? 8 : 16;
  dma_barrier<kWaitFirst>();  // tile 0 has landed
  // Fragments are read one whole tile ahead: fa/fb[set][ks][block], the
  // set alternating with the tile's parity.
  bf16x8 fa[2][2][4], fb[2][2][4];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa[0][ks][i] = frag<AK>(ra + tile_base<AK, NSA>(0), oa, i, 0, ks);
      fb[0][ks][i] = frag<BKC>(rb + tile_base<BKC, NSB>(0), ob, i, 0, ks);
    }
  // Tile kt: one barrier at the top, then 32 MFMAs on fragments in hand;
  // next to the first 16 the 16 fragment reads of tile kt+1, and the loads,
  // A's before B's: a k-contiguous A with three slots loads half of its pair
  // kt+5, kt+6 (odd kt) or the other half of pair kt+4, kt+5 (even kt), with
  // two slots its pair kt+3, kt+4 (odd kt); a k-contiguous B its pair kt+3,
  // kt+4 (odd kt); an mn-contiguous operand its tile kt+4.  At the barrier
  // tile kt+1 must have landed; only loads issued after its last one may
  // still be in flight.
  auto tile = [&](auto parity, int kt) {
    constexpr int P = decltype(parity)::value;  // kt % 2
    const bf16* na = ra + tile_base<AK, NSA>(kt + 1);
    const bf16* nb = rb + tile_base<BKC, NSB>(kt + 1);
    dma_barrier<P == 0 ? kWaitEven : kWaitOdd>();
#pragma unroll
    for (int q = 0; q < 32; ++q) {
      const int ks = q >> 4, i = (q >> 2) & 3, j = q & 3;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[P][ks][j], fa[P][ks][i], acc[i][j], 0, 0, 0);
      if (q < 16) {  // read order per k-substep: B0 A0 B1 B2 B3 A1 A2 A3
        const int rk = q >> 3, r = q & 7;
        if (r == 0 || r == 2 || r == 3 || r == 4)
          fb[P ^ 1][rk][r == 0 ? 0 : r - 1] = frag<BKC>(nb, ob, r == 0 ? 0 : r - 1, P ^ 1, rk);
        else
          fa[P ^ 1][rk][r == 1 ? 0 : r - 4] = frag<AK>(na, oa, r == 1 ? 0 : r - 4, P ^ 1, rk);
      }
      if constexpr (NSA == 3) {
        if (q < 8 && (q & 1) == 0) load_a(P == 1 ? kt + 5 : kt + 4, (P == 1 ? 0 : 4) + (q >> 1));
      } else if constexpr (AK) {
        if (P == 1 && q < 16 && (q & 1)) load_a(kt + 3, q >> 1);
      } else {
        if (q < 16 && (q & 3) == 3) load_a(kt + 4, q >> 2);
      }
      if constexpr (BKC) {
        constexpr int q0 = AK ? 8 : 16;  // after A's loads
        if (P == 1 && q >= q0 && q < q0 + kLoadsKC) load_b(kt + 3, q - q0);
      } else {
        if (q >= 16 && (q & 3) == 3) load_b(kt + 4, (q - 16) >> 2);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Tiles in pairs (a phantom tile past the end loads and multiplies zeros).
  for (int kt = 0; kt < nk; kt += 2) {
    tile(std::integral_constant<int, 0>(), kt);
    tile(std::integral_constant<int, 1>(), kt + 1);
  }

  // Epilogue staged through LDS.  A lane holds, per 32x32 block, one output
  // row and 4 consecutive columns; stored directly that scatters every store
  // over 32 rows.  Instead each wave writes one block row of its results
  // (32 x 128 float32, alpha applied) into a private [32][kStagePitch] block
  // and reads it back row-major: a half-wave then covers 128 contiguous
  // columns of one row, so the residual loads and the output stores (one
  // rounding, after the residual) are fully coalesced.  The blocks are
  // private to the wave, so after one barrier (the ring's last loads have
  // landed everywhere) only the wave's own LDS accesses are ordered: no
  // workgroup barrier, whose memory fence would wait for every store in
  // flight, and the stores drain while the wave goes on.
  const float alpha = g.alpha * (g.alpha_dev ? *g.alpha_dev : 1.f);
  const int half = lane >> 5, lm = lane & 31;
  float* part = g.part ? g.part + static_cast<int64_t>(sp) * g.M * g.N : nullptr;
  float* stage = reinterpret_cast<float*>(ring) + wave * (32 * kStagePitch);
  const int c = lm * 4;
  const int n = n0 + wn * 128 + c;
  // A block row takes the branch-free path when all its 32 rows and 128
  // columns are in range.
  const bool full_cols = n0 + wn * 128 + 128 <= g.N;
  // Largest kept sequence index, for the row map (rows < M only).
  const int q_last = g.out_map.idx && M > 0 ? (M - 1) / g.out_map.S : 0;
  dma_barrier<0>();  // the loop's last loads (zeros) land before the ring is reused
  // A plain bf16 output (no residual, row map or partials) is rounded as it
  // is staged: half the LDS traffic, and 16-byte stores that cover a row's
  // 128 columns with 16 lanes (four rows per instruction).  The same single
  // rounding of alpha * acc as the float32 staging gives.  Block rows that
  // cross M store straight from the accumulators, row by row.
  if constexpr (EPI == kEpiGluFwd) {
    // [u v] and s are bf16 outputs too, staged as bf16 the same way; rows
    // past M are not stored
    {
      bf16* st16 = reinterpret_cast<bf16*>(stage);
      const int rr = lane >> 4, cc = (lane & 15) * 8;  // [u v]: row rr of each 4, columns cc..cc+7
      const int rs = lane >> 3, cs = (lane & 7) * 8;   // s: row rs of each 8, columns cs..cs+7
      const int f0 = tn * 128 + wn * 64;               // the wave's first d_ff column
      bf16* C = static_cast<bf16*>(g.C);
      bf16* Sp = static_cast<bf16*>(g.aux);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mb = m0 + wm * 128 + i * 32;
        if (mb >= M) break;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const floatx16& a = acc[i][j];
            *reinterpret_cast<uint2*>(st16 + lm * kStagePitch16 + j * 32 + 8 * q + 4 * half) =
                pack4_bf16(alpha * a[4 * q], alpha * a[4 * q + 1], alpha * a[4 * q + 2], alpha * a[4 * q + 3]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        // staged columns 0-63 are gate (u) columns, 64-127 up (v) columns
        const int gcol = cc < 64 ? f0 + cc : g.glu_f + f0 + cc - 64;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const bf16* src = st16 + (4 * k + rr) * kStagePitch16 + cc;
          const uint2 lo = *reinterpret_cast<const uint2*>(src), hi = *reinterpret_cast<const uint2*>(src + 4);
          if (mb + 4 * k + rr < M)
            *reinterpret_cast<uint4*>(C + static_cast<int64_t>(mb + 4 * k + rr) * g.ldc + gcol) =
                make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        // s = silu(u) v from the float32 accumulators (see below)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float sv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              sv[e] = swiglu_fwd_f(alpha * acc[i][j][4 * q + e], alpha * acc[i][j + 2][4 * q + e]);
            *reinterpret_cast<uint2*>(st16 + lm * kStagePitch16 + j * 32 + 8 * q + 4 * half) =
                pack4_bf16(sv[0], sv[1], sv[2], sv[3]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bf16* src = st16 + (8 * k + rs) * kStagePitch16 + cs;
          const uint2 lo = *reinterpret_cast<const uint2*>(src), hi = *reinterpret_cast<const uint2*>(src + 4);
          if (mb + 8 * k + rs < M)
            *reinterpret_cast<uint4*>(Sp + static_cast<int64_t>(mb + 8 * k + rs) * g.glu_f + f0 + cs) =
                make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // reads done before the block is rewritten
      }
      return;
    }
  }
  if constexpr (EPI == kEpiPlain) {
    if (!part && !g.R && !g.c_f32 && !g.out_map.idx && full_cols) {
      bf16* st16 = reinterpret_cast<bf16*>(stage);
      const int rr = lane >> 4, cc = (lane & 15) * 8;  // read: row rr of each 4, columns cc..cc+7
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mb = m0 + wm * 128 + i * 32;
        if (mb + 32 > M) {
          if (mb < M) epilogue_plain_edge_bf16(g, acc[i], alpha, mb, n0 + wn * 128, lm, half, M);
          continue;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const floatx16& a = acc[i][j];
            *reinterpret_cast<uint2*>(st16 + lm * kStagePitch16 + j * 32 + 8 * q + 4 * half) =
                pack4_bf16(alpha * a[4 * q], alpha * a[4 * q + 1], alpha * a[4 * q + 2], alpha * a[4 * q + 3]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        // rows are 264 bytes apart (8-byte aligned, no bank conflicts for the
        // 8-byte stage writes), so each 16 bytes are read as two 8-byte halves
        uint4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const bf16* src = st16 + (4 * k + rr) * kStagePitch16 + cc;
          const uint2 lo = *reinterpret_cast<const uint2*>(src), hi = *reinterpret_cast<const uint2*>(src + 4);
          v[k] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
        bf16* C = static_cast<bf16*>(g.C);
#pragma unroll
        for (int k = 0; k < 8; ++k)
          *reinterpret_cast<uint4*>(C + static_cast<int64_t>(mb + 4 * k + rr) * g.ldc + n0 + wn * 128 + cc) = v[k];
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // reads done before the block is rewritten
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const floatx16& a = acc[i][j];
        *reinterpret_cast<float4*>(stage + lm * kStagePitch + j * 32 + 8 * q + 4 * half) =
            make_float4(alpha * a[4 * q], alpha * a[4 * q + 1], alpha * a[4 * q + 2], alpha * a[4 * q + 3]);
      }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // staged values visible to the wave
    const int mb = m0 + wm * 128 + i * 32;             // first row of the block row
    if constexpr (EPI == kEpiGluBwd) {
      glu_bwd_rows(g, stage, mb + half, half, c, n, M, n0 + wn * 128 + 128 <= g.N && mb + 32 <= M);
    } else if constexpr (EPI == kEpiRelu2Fwd) {
      relu2_fwd_rows(g, stage, mb + half, half, c, n, M, n0 + wn * 128 + 128 <= g.N && mb + 32 <= M);
    } else if constexpr (EPI == kEpiRelu2Bwd) {
      relu2_bwd_rows(g, stage, mb + half, half, c, n, M, n0 + wn * 128 + 128 <= g.N && mb + 32 <= M);
    } else {
      if (full_cols && mb + 32 <= M)
        epilogue_rows_full(g, part, stage, mb + half, half, c, n, q_last);
      else
        epilogue_rows_edge(g, part, stage, mb + half, half, c, n, M);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // reads done before the block is rewritten
  }
}

#define LD_BIG_ATTRS __global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
#define LD_BIG_KERNEL(name, ak, bk)                                                    \
  LD_BIG_ATTRS void name(GemmArgs g) {                                                 \
    __shared__ __align__(16) bf16 ring[ring_elems<ak, bk>()];                          \
    gemm_big_body<ak, bk>(g, ring, blockIdx.x, gridDim.x, blockIdx.y, gridDim.y);      \
  }
LD_BIG_KERNEL(ld_gemm_bf16_nt_256, true, true)
LD_BIG_KERNEL(ld_gemm_bf16_nn_256, true, false)
LD_BIG_KERNEL(ld_gemm_bf16_tn_256, false, false)
LD_BIG_KERNEL(ld_gemm_bf16_tt_256, false, true)

// C = [u v] rows and aux = silu(u) v rows of the SwiGLU projection (see GemmArgs).
LD_BIG_ATTRS void ld_gemm_bf16_nt_glu_256(GemmArgs g) {
  __shared__ __align__(16) bf16 ring[ring_elems<true, true>()];
  gemm_big_body<true, true, kEpiGluFwd>(g, ring, blockIdx.x, gridDim.x, 0, 1);
}

// C = u rows and aux = relu(u)^2 rows of the squared-ReLU projection (see GemmArgs).
LD_BIG_ATTRS void ld_gemm_bf16_nt_relu2_256(GemmArgs g) {
  __shared__ __align__(16) bf16 ring[ring_elems<true, true>()];
  gemm_big_body<true, true, kEpiRelu2Fwd>(g, ring, blockIdx.x, gridDim.x, 0, 1);
}

// Up to three GEMMs in one launch: weight-gradient GEMMs g1 (tiles1 tiles,
// each split into splits1 k ranges) and g3 (tiles3 tiles, never split; both
// with both operands mn-contiguous) and an input-gradient GEMM g2 (A
// k-contiguous, B mn-contiguous, tiles2 tiles).  The workgroups go in the
// order g3, g1, g2, or g2 first (g2_first); the later GEMMs' workgroups
// fill the CUs the earlier ones leave idle, so no GEMM's last partial round
// runs on a part-empty chip.  tiles1 = tiles3 = 0 leaves g2 alone.
template <int EPI2>
__device__ __forceinline__ void gemm_pair_body(const GemmArgs& g1, const GemmArgs& g3, const GemmArgs& g2, int tiles1,
                                               int splits1, int tiles3, int tiles2, int g2_first) {
  __shared__ __align__(16) bf16 ring[ring_elems<true, false>()];
  const int n1 = tiles1 * splits1;
  int id = blockIdx.x;
  if (g2_first) {
    if (id < tiles2) {
      gemm_big_body<true, false, EPI2>(g2, ring, id, tiles2, 0, 1);
      return;
    }
    id -= tiles2;
  } else if (id >= tiles3 + n1) {
    gemm_big_body<true, false, EPI2>(g2, ring, id - tiles3 - n1, tiles2, 0, 1);
    return;
  }
  if (id < tiles3)
    gemm_big_body<false, false>(g3, ring, id, tiles3, 0, 1);
  else
    gemm_big_body<false, false>(g1, ring, (id - tiles3) % tiles1, tiles1, (id - tiles3) / tiles1, splits1);
}
LD_BIG_ATTRS void ld_gemm_bf16_tn_nn_256(GemmArgs g1, GemmArgs g3, GemmArgs g2, int tiles1, int splits1, int tiles3,
                                         int tiles2, int g2_first) {
  gemm_pair_body<kEpiPlain>(g1, g3, g2, tiles1, splits1, tiles3, tiles2, g2_first);
}
// The same with the SwiGLU backward fused into g2's epilogue (see GemmArgs).
LD_BIG_ATTRS void ld_gemm_bf16_tn_nn_glu_256(GemmArgs g1, GemmArgs g3, GemmArgs g2, int tiles1, int splits1,
                                             int tiles3, int tiles2, int g2_first) {
  gemm_pair_body<kEpiGluBwd>(g1, g3, g2, tiles1, splits1, tiles3, tiles2, g2_first);
}
// The same with the squared-ReLU backward fused into g2's epilogue.
LD_BIG_ATTRS void ld_gemm_bf16_tn_nn_relu2_256(GemmArgs g1, GemmArgs g3, GemmArgs g2, int tiles1, int splits1,
                                               int tiles3, int tiles2, int g2_first) {
  gemm_pair_body<kEpiRelu2Bwd>(g1, g3, g2, tiles1, splits1, tiles3, tiles2, g2_first);
}

// C[i] = sum over splits of part[s][i], float32, in split order.  Every
// split's value is requested before the first add (splits <= kMaxSplits).
constexpr int kMaxSplits = 8;
__global__ __launch_bounds__(256) void ld_splitk_reduce(const float* part, int splits, int64_t mn, float* C) {
  for (int64_t i4 = blockIdx.x * 256ll + threadIdx.x; i4 < mn / 4; i4 += gridDim.x * 256ll) {
    float4 t[kMaxSplits];
#pragma unroll
    for (int k = 0; k < kMaxSplits; ++k)
      if (k < splits) t[k] = reinterpret_cast<const float4*>(part + static_cast<int64_t>(k) * mn)[i4];
    float4 sum = t[0];
#pragma unroll
    for (int k = 1; k < kMaxSplits; ++k)
      if (k < splits) {
        sum.x += t[k].x; sum.y += t[k].y; sum.z += t[k].z; sum.w += t[k].w;
      }
    reinterpret_cast<float4*>(C)[i4] = sum;
  }
}

// Dynamic LDS limit of the 128x128 kernels, raised once per process (a
// function-local static: its initialisation is thread-safe).
void set_attrs() {
  static const bool done = [] {
    const void* small[] = {reinterpret_cast<const void*>(ld_gemm_bf16_nt),
                           reinterpret_cast<const void*>(ld_gemm_bf16_nn),
                           reinterpret_cast<const void*>(ld_gemm_bf16_tn),
                           reinterpret_cast<const void*>(ld_gemm_bf16_tt)};
    for (const void* f : small) (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
    return true;
  }();
  (void)done;
}

}  // namespace

GemmPlan plan_gemm(int dtype, int a_kcontig, int b_kcontig, const GemmArgs& g, int64_t max_m,
                   int64_t max_k, bool allow_split) {
  GemmPlan p{};
  p.splits = 1;
  if (dtype != LD_BF16) {
    p.name = "ld_gemm_f32_k";
    return p;
  }
  const int64_t big_tiles = ((max_m + GB - 1) / GB) * ((g.N + GB - 1) / GB);
  // the big tile's epilogue stores 4 consecutive columns at once
  // each operand is addressed through one buffer descriptor: spans < 2 GiB
  const int64_t a_span = 2 * g.lda * (a_kcontig ? max_m : max_k);
  const int64_t b_span = 2 * g.ldb * (b_kcontig ? static_cast<int64_t>(g.N) : max_k);
  // split-K only for float32 outputs without a residual (weight gradients);
  // such a GEMM fills the CUs through its splits even with few tiles
  const bool splittable = allow_split && g.c_f32 && !g.R && !g.out_map.idx && g.ldc == g.N && max_k >= 16 * GK;
  p.big = (g.N % 4 == 0) && (g.ldc % 4 == 0) && (!g.R || g.ldr % 4 == 0) && max_m >= 512 && g.N >= 512 &&
          (big_tiles >= 32 || (splittable && big_tiles * kMaxSplits >= 32)) && a_span < kBigMaxSpan &&
          b_span < kBigMaxSpan;
  if (p.big) {
    if (splittable) {
      double best = 0;
      for (int s = 1; s <= kMaxSplits; ++s) {
        const int64_t wg = big_tiles * s;
        const double eff = static_cast<double>(wg) / (256.0 * ((wg + 255) / 256)) - 0.02 * (s - 1);
        if (eff > best + 1e-9 && max_k / s >= 8 * GK) {
          best = eff;
          p.splits = s;
        }
      }
    }
    p.name = a_kcontig && b_kcontig ? "ld_gemm_bf16_nt_256"
             : a_kcontig            ? "ld_gemm_bf16_nn_256"
             : b_kcontig            ? "ld_gemm_bf16_tt_256"
                                    : "ld_gemm_bf16_tn_256";
  } else {
    p.name = a_kcontig && b_kcontig ? "ld_gemm_bf16_nt"
             : a_kcontig            ? "ld_gemm_bf16_nn"
             : b_kcontig            ? "ld_gemm_bf16_tt"
                                    : "ld_gemm_bf16_tn";
  }
  return p;
}

size_t gemm_part_bytes(const GemmPlan& p, int64_t M, int64_t N) {
  return p.splits > 1 ? 4ull * p.splits * M * N : 0;
}

const char* gemm_kernel_name(int dtype, int a_kcontig, int b_kcontig) {
  if (dtype == LD_BF16) {
    if (a_kcontig && b_kcontig) return "ld_gemm_bf16_nt";
    if (a_kcontig) return "ld_gemm_bf16_nn";
    if (b_kcontig) return "ld_gemm_bf16_tt";
    return "ld_gemm_bf16_tn";
  }
  return "ld_gemm_f32_k";
}

hipError_t launch_gemm_plan(int dtype, int a_kcontig, int b_kcontig, const GemmPlan& p, GemmArgs g,
                            int64_t max_m, hipStream_t s) {
  if (max_m <= 0 || g.N <= 0) return hipSuccess;
  if (dtype == LD_BF16 && p.big) {
    set_attrs();
    const int64_t tiles = ((max_m + GB - 1) / GB) * ((g.N + GB - 1) / GB);
    float* C = static_cast<float*>(g.C);
    if (p.splits > 1) {
      if (!g.part) return hipErrorInvalidValue;
    } else {
      g.part = nullptr;
    }
    const dim3 grid(static_cast<unsigned>(tiles), p.splits), block(256);
    if (a_kcontig && b_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_nt_256, grid, block, 0, s, g);
    else if (a_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_nn_256, grid, block, 0, s, g);
    else if (b_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_tt_256, grid, block, 0, s, g);
    else
      hipLaunchKernelGGL(ld_gemm_bf16_tn_256, grid, block, 0, s, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t mn = static_cast<int64_t>(g.M) * g.N;
    int blocks = static_cast<int>(std::min<int64_t>((mn / 4 + 255) / 256, 1 << 20));
    hipLaunchKernelGGL(ld_splitk_reduce, dim3(blocks), dim3(256), 0, s, g.part, p.splits, mn, C);
    return hipGetLastError();
  }
  return launch_gemm(dtype, a_kcontig, b_kcontig, g, max_m, 0, s);
}

// Estimated finish time, in k tiles of 32 (~1 us each at these shapes), of
// classes of workgroups (count, cost each) dealt in launch order to n_cu
// CUs, one workgroup per CU, each CU taking the next when it frees.
static double list_schedule(std::initializer_list<std::pair<int64_t, double>> classes, int n_cu) {
  std::priority_queue<double, std::vector<double>, std::greater<double>> cu;
  for (int i = 0; i < n_cu; ++i) cu.push(0.0);
  double end = 0.0;
  for (const auto& c : classes)
    for (int64_t w = 0; w < c.first; ++w) {
      const double t = cu.top() + c.second;
      cu.pop();
      cu.push(t);
      end = std::max(end, t);
    }
  return end;
}

PairPlan plan_gemm_pair(int64_t m1, int64_t n1, int64_t k1, int64_t m3, int64_t n3, int64_t m2, int64_t n2,
                        int64_t k2, int max_splits) {
  int dev = 0, n_cu = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (n_cu <= 0) n_cu = 256;
  struct Entry {
    int64_t key[9];
    PairPlan plan;
  };
  constexpr int kEntries = 64;  // the kept counts of a step give a few dozen shapes
  thread_local Entry cache[kEntries];
  thread_local int next = 0;
  const int64_t key[9] = {m1, n1, k1, m3, n3, m2, n2, k2, max_splits * 4096ll + n_cu};
  for (const Entry& e : cache)
    if (std::equal(key, key + 9, e.key)) return e.plan;
  constexpr double kEpi = 8.0;       // epilogue of one tile, in k-tile times
  constexpr double kLaunch = 4.0;    // a second (reduction) launch
  constexpr double kTileUs = 0.95;   // one k tile of 32 on one CU
  auto tiles = [](int64_t m, int64_t n) { return ((m + GB - 1) / GB) * ((n + GB - 1) / GB); };
  const int64_t tiles1 = m1 > 0 ? tiles(m1, n1) : 0, tiles3 = m3 > 0 ? tiles(m3, n3) : 0;
  const int64_t tiles2 = tiles(m2, n2);
  const int64_t nkt1 = (k1 + GK - 1) / GK;
  const double c2 = static_cast<double>((k2 + GK - 1) / GK) + kEpi;
  const double c3 = static_cast<double>(nkt1) + kEpi;
  PairPlan best{1, 0, 0.0};
  double best_t = 0.0;
  for (int sp = 1; sp <= (tiles1 > 0 ? max_splits : 1); ++sp) {
    const double c1 = static_cast<double>((nkt1 + sp - 1) / sp) + kEpi;
    for (int order = 0; order < 2; ++order) {
      double t = order ? list_schedule({{tiles2, c2}, {tiles3, c3}, {tiles1 * sp, c1}}, n_cu)
                       : list_schedule({{tiles3, c3}, {tiles1 * sp, c1}, {tiles2, c2}}, n_cu);
      if (sp > 1)  // partials written and read back at ~5 TB/s, plus a launch
        t += kLaunch + (sp + 1.0) * 4.0 * m1 * n1 / 5e12 / (kTileUs * 1e-6);
      if ((sp == 1 && order == 0) || t < best_t - 1e-9) {
        best_t = t;
        best = PairPlan{sp, order, t};
      }
    }
  }
  Entry& e = cache[next];
  next = (next + 1) % kEntries;
  std::copy(key, key + 9, e.key);
  e.plan = best;
  return best;
}

hipError_t launch_gemm_glu_fwd(const GemmArgs& g, int64_t max_m, hipStream_t s) {
  if (max_m <= 0 || g.N <= 0) return hipSuccess;
  const int64_t tiles = ((max_m + GB - 1) / GB) * (g.N / GB);
  hipLaunchKernelGGL(ld_gemm_bf16_nt_glu_256, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_gemm_relu2_fwd(const GemmArgs& g, int64_t max_m, hipStream_t s) {
  if (max_m <= 0 || g.N <= 0) return hipSuccess;
  const int64_t tiles = ((max_m + GB - 1) / GB) * ((g.N + GB - 1) / GB);
  hipLaunchKernelGGL(ld_gemm_bf16_nt_relu2_256, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_gemm_pair(GemmArgs g1, const GemmArgs* g3, const PairPlan& p, const GemmArgs& g2, int64_t max_m2,
                            hipStream_t s) {
  const int splits1 = p.splits1;
  const int64_t tiles1 =
      g1.M > 0 ? ((static_cast<int64_t>(g1.M) + GB - 1) / GB) * ((g1.N + GB - 1) / GB) : 0;
  const int64_t tiles3 =
      g3 ? ((static_cast<int64_t>(g3->M) + GB - 1) / GB) * ((g3->N + GB - 1) / GB) : 0;
  const int64_t tiles2 = ((max_m2 + GB - 1) / GB) * ((g2.N + GB - 1) / GB);
  if (splits1 > 1) {
    if (!g1.part) return hipErrorInvalidValue;
  } else {
    g1.part = nullptr;
  }
  const GemmArgs g3v = g3 ? *g3 : g1;
  const int64_t wg = tiles1 * splits1 + tiles3 + tiles2;
  if (wg <= 0) return hipSuccess;
  if (g2.relu2)
    hipLaunchKernelGGL(ld_gemm_bf16_tn_nn_relu2_256, dim3(static_cast<unsigned>(wg)), dim3(256), 0, s, g1, g3v, g2,
                       static_cast<int>(tiles1), splits1, static_cast<int>(tiles3), static_cast<int>(tiles2),
                       p.g2_first);
  else if (g2.glu_f > 0)
    hipLaunchKernelGGL(ld_gemm_bf16_tn_nn_glu_256, dim3(static_cast<unsigned>(wg)), dim3(256), 0, s, g1, g3v, g2,
                       static_cast<int>(tiles1), splits1, static_cast<int>(tiles3), static_cast<int>(tiles2),
                       p.g2_first);
  else
    hipLaunchKernelGGL(ld_gemm_bf16_tn_nn_256, dim3(static_cast<unsigned>(wg)), dim3(256), 0, s, g1, g3v, g2,
                       static_cast<int>(tiles1), splits1, static_cast<int>(tiles3), static_cast<int>(tiles2),
                       p.g2_first);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, int splits, int64_t mn, float* C, hipStream_t s) {
  if (splits <= 1 || mn <= 0) return hipSuccess;
  const int blocks = static_cast<int>(std::min<int64_t>((mn / 4 + 255) / 256, 1 << 20));
  hipLaunchKernelGGL(ld_splitk_reduce, dim3(blocks), dim3(256), 0, s, part, splits, mn, C);
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int a_kcontig, int b_kcontig, const GemmArgs& g, int64_t max_m,
                       int64_t max_k, hipStream_t s) {
  (void)max_k;
  if (max_m <= 0 || g.N <= 0) return hipSuccess;
  if (dtype == LD_BF16) {
    set_attrs();
    const int64_t tiles = ((max_m + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    const dim3 grid(static_cast<unsigned>(tiles)), block(256);
    if (a_kcontig && b_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_nt, grid, block, kGemmLds, s, g);
    else if (a_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_nn, grid, block, kGemmLds, s, g);
    else if (b_kcontig)
      hipLaunchKernelGGL(ld_gemm_bf16_tt, grid, block, kGemmLds, s, g);
    else
      hipLaunchKernelGGL(ld_gemm_bf16_tn, grid, block, kGemmLds, s, g);
    return hipGetLastError();
  }
  const int64_t tiles = ((max_m + FT - 1) / FT) * ((g.N + FT - 1) / FT);
  const dim3 grid(static_cast<unsigned>(tiles)), block(256);
  if (a_kcontig && b_kcontig)
    hipLaunchKernelGGL((ld_gemm_f32_k<true, true>), grid, block, 0, s, g);
  else if (a_kcontig)
    hipLaunchKernelGGL((ld_gemm_f32_k<true, false>), grid, block, 0, s, g);
  else if (b_kcontig)
    hipLaunchKernelGGL((ld_gemm_f32_k<false, true>), grid, block, 0, s, g);
  else
    hipLaunchKernelGGL((ld_gemm_f32_k<false, false>), grid, block, 0, s, g);
  return hipGetLastError();
}

}  // namespace ld

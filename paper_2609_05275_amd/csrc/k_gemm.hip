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
    if (g.c_f32)
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

bool g_attr_done = false;

}  // namespace

const char* gemm_kernel_name(int dtype, int a_kcontig, int b_kcontig) {
  if (dtype == LD_BF16) {
    if (a_kcontig && b_kcontig) return "ld_gemm_bf16_nt";
    if (a_kcontig) return "ld_gemm_bf16_nn";
    if (b_kcontig) return "ld_gemm_bf16_tt";
    return "ld_gemm_bf16_tn";
  }
  return "ld_gemm_f32_k";
}

hipError_t launch_gemm(int dtype, int a_kcontig, int b_kcontig, const GemmArgs& g, int64_t max_m,
                       int64_t max_k, hipStream_t s) {
  (void)max_k;
  if (max_m <= 0 || g.N <= 0) return hipSuccess;
  if (dtype == LD_BF16) {
    if (!g_attr_done) {
      hipFuncSetAttribute(reinterpret_cast<const void*>(ld_gemm_bf16_nt),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
      hipFuncSetAttribute(reinterpret_cast<const void*>(ld_gemm_bf16_nn),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
      hipFuncSetAttribute(reinterpret_cast<const void*>(ld_gemm_bf16_tn),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
      hipFuncSetAttribute(reinterpret_cast<const void*>(ld_gemm_bf16_tt),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
      g_attr_done = true;
    }
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

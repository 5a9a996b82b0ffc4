// Kernels of incremental (KV-cached) decoding: a few new rows per sequence
// go through a layer whose keys and values of earlier positions are cached.
// Both hot kernels are bound by HBM reads: the skinny GEMM reads each weight
// matrix once, the decode attention reads each cached key/value row once.
//
// Skinny GEMM (M <= 64 rows, bf16, v_mfma_f32_32x32x16_bf16): one wave owns
// 32 output columns; the four waves of a workgroup (and, with ksplit > 1,
// several workgroups) take interleaved 64-wide k chunks of the same columns.
// Within a chunk the k index of the four MFMAs is permuted so that each lane
// reads 64 contiguous bytes of its row: lane half h, MFMA s holds
// k = 64c + 32h + 8s + e (e < 8), in A and W alike, which leaves the
// contraction unchanged.  The waves' accumulators are summed in LDS in wave
// order; split workgroups write float32 partials summed in split order by a
// second kernel, so results do not depend on timing.  (A last-arriving
// workgroup doing that sum needs device-scope fences, which on this chip
// write back and invalidate the per-XCD L2 and cost far more than the
// second launch.)
//
// Decode attention: one workgroup per (256-key chunk, head, sequence), a
// wave per 64 keys.  Scores in base 2 with the causal cut (key <= query
// position) and the ALiBi bias: for one query row, dh/8 lanes per key, each
// with 8 of the head's dimensions, summed by lane exchanges; for several
// rows, S^T = K Q^T on the matrix cores (the rows padded to 32 columns).
// Softmax statistics per query row over the chunk, then P V with dh/8 lanes
// per key (16-byte coalesced value reads), summed over the wave's keys by
// lane exchanges and over the four waves in LDS.  A combine kernel merges
// the chunks with the usual max/sum rescaling and writes bf16.
#include "ld_internal.h"

namespace ld {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kSkWaves = 4;
constexpr int kSkChunk = 64;

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = static_cast<bf16>(0.f);
  return z;
}

__device__ __forceinline__ bf16x8 load8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ void skinny_store(const SkinnyArgs& g, int m, int n, float sum) {
  float v = g.alpha * sum;
  if (g.R) v += static_cast<float>(static_cast<const bf16*>(g.R)[static_cast<int64_t>(m) * g.ldr + n]);
  const bf16 o = static_cast<bf16>(v);
  static_cast<bf16*>(g.C)[static_cast<int64_t>(m) * g.ldc + n] = o;
  if (g.kv && n >= g.kv_d) {
    const int64_t b = m / g.kv_n, j = m % g.kv_n;
    static_cast<bf16*>(g.kv)[(b * g.kv_s_max + g.kv_pos + j) * 2 * g.kv_d + (n - g.kv_d)] = o;
  }
}

template <int MB>
__global__ __launch_bounds__(256) void ld_gemm_bf16_skinny(SkinnyArgs g) {
  __shared__ float red[kSkWaves * MB * 16 * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 31, h = lane >> 5;
  const int n0 = blockIdx.x * 32;
  const int nchunks = (g.K + kSkChunk - 1) / kSkChunk;
  const int workers = kSkWaves * gridDim.y;
  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* W = static_cast<const bf16*>(g.W);
  const bool nvalid = n0 + li < g.N;
  const bf16* wrow = W + static_cast<int64_t>(nvalid ? n0 + li : 0) * g.ldw + 32 * h;
  const bf16* arow[MB];
  bool mvalid[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    mvalid[mb] = mb * 32 + li < g.M;
    arow[mb] = A + static_cast<int64_t>(mvalid[mb] ? mb * 32 + li : 0) * g.lda + 32 * h;
  }
  floatx16 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;

  // U chunks per pass, all loaded before their MFMAs (chunks past the end
  // load zeros, so the MFMAs need no branch)
  constexpr int U = MB == 1 ? 4 : 2;
  for (int c0 = blockIdx.y * kSkWaves + wave; c0 < nchunks; c0 += U * workers) {
    bf16x8 b[U][4], a[U][MB][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kc = (c0 + u * workers) * kSkChunk;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bool kv = kc + 32 * h + 8 * s < g.K;   // K % 8 == 0: the whole 8 are in range
        b[u][s] = (nvalid && kv) ? load8(wrow + kc + 8 * s) : zero8();
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          a[u][mb][s] = (mvalid[mb] && kv) ? load8(arow[mb] + kc + 8 * s) : zero8();
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[u][mb][s], b[u][s], acc[mb], 0, 0, 0);
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) red[((wave * MB + mb) * 16 + v) * 64 + lane] = acc[mb][v];
  __syncthreads();
  constexpr int kElems = MB * 16 * 64;
  for (int e = threadIdx.x; e < kElems; e += 256) {
    float sum = red[e];
#pragma unroll
    for (int w = 1; w < kSkWaves; ++w) sum += red[w * kElems + e];
    const int l = e & 63, v = (e >> 6) & 15, mb = e >> 10;
    const int m = mb * 32 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
    const int n = n0 + (l & 31);
    if (m < g.M && n < g.N) {
      if (gridDim.y > 1 || g.part_only)
        g.part[(static_cast<int64_t>(blockIdx.y) * g.M + m) * g.N + n] = sum;
      else
        skinny_store(g, m, n, sum);
    }
  }
}

__global__ __launch_bounds__(256) void ld_skinny_reduce_k(SkinnyArgs g, int ksplit) {
  const int64_t total = static_cast<int64_t>(g.M) * g.N;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < total; i += gridDim.x * 256ll) {
    float sum = g.part[i];
    for (int s = 1; s < ksplit; ++s) sum += g.part[s * total + i];
    skinny_store(g, static_cast<int>(i / g.N), static_cast<int>(i % g.N), sum);
  }
}

__device__ __forceinline__ float bf16r(float x) { return static_cast<float>(static_cast<bf16>(x)); }

// Split-K sums (split order) of one row of a skinny GEMM with alpha and the
// residual, stored as C, then (when a gain is given) the RMSNorm of the
// stored row (sum of squares over the workgroup in a fixed order):
// h = bf16(C rstd gain).  One workgroup of 1024 threads per row.
__global__ __launch_bounds__(1024) void ld_skinny_reduce_norm_k(SkinnyArgs g, int ksplit, const bf16* gain,
                                                                 float eps, bf16* h) {
  constexpr int kPer = 4;  // columns per thread and pass: one pass up to 4096 columns
  __shared__ float wsum[16];
  const int m = blockIdx.x, tid = threadIdx.x;
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  const float* prow = g.part + static_cast<int64_t>(m) * g.N;
  bf16* C = static_cast<bf16*>(g.C) + static_cast<int64_t>(m) * g.ldc;
  const bf16* R = g.R ? static_cast<const bf16*>(g.R) + static_cast<int64_t>(m) * g.ldr : nullptr;
  float ss = 0.f;
  for (int n0 = 0; n0 < g.N; n0 += 1024 * kPer) {
    float sum[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) sum[i] = 0.f;
    // the splits in order; every column's loads of a split are independent
#pragma unroll 2
    for (int sp = 0; sp < ksplit; ++sp)
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int n = n0 + i * 1024 + tid;
        if (n < g.N) sum[i] += prow[sp * mn + n];
      }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int n = n0 + i * 1024 + tid;
      if (n < g.N) {
        const bf16 o = static_cast<bf16>(g.alpha * sum[i] + (R ? static_cast<float>(R[n]) : 0.f));
        C[n] = o;
        const float of = static_cast<float>(o);
        ss = __builtin_fmaf(of, of, ss);
      }
    }
  }
  if (!gain) return;  // no norm follows (workgroup-uniform)
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, 64);
  if ((tid & 63) == 0) wsum[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += wsum[w];
  const float rstd = rsqrtf(tot / static_cast<float>(g.N) + eps);
  bf16* hr = h + static_cast<int64_t>(m) * g.N;
  for (int n = tid; n < g.N; n += 1024)  // this thread's own stores, read back
    hr[n] = static_cast<bf16>(static_cast<float>(C[n]) * rstd * static_cast<float>(gain[n]));
}

// The FFN activation from a skinny GEMM's partials: u (and v = column f + n
// for SwiGLU) rounded to bf16 as stored outputs would be, s = act(u, v).
__global__ __launch_bounds__(256) void ld_skinny_reduce_act_k(SkinnyArgs g, int ksplit, int act, int f, bf16* so) {
  const int64_t mn = static_cast<int64_t>(g.M) * g.N, total = static_cast<int64_t>(g.M) * f;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < total; i += gridDim.x * 256ll) {
    const int64_t m = i / f, n = i % f, iu = m * g.N + n;
    float su = g.part[iu];
#pragma unroll 4
    for (int sp = 1; sp < ksplit; ++sp) su += g.part[sp * mn + iu];
    const float u = bf16r(g.alpha * su);
    float out;
    if (act == kDecActSwiglu) {
      float sv = g.part[iu + f];
#pragma unroll 4
      for (int sp = 1; sp < ksplit; ++sp) sv += g.part[sp * mn + iu + f];
      out = swiglu_fwd_f(u, bf16r(g.alpha * sv));
    } else {
      const float z = fmaxf(u, 0.f);
      out = z * z;
    }
    so[m * f + n] = static_cast<bf16>(out);
  }
}

// ------------------------------------------------ fused decode projection
// At most 8 rows, so the product is a few dot products per weight: vector
// ALU work (v_dot2 on bf16 pairs), not MFMA tiles, and the layout is chosen
// for the weight stream.  A tile is 8 output columns (8 rows of W; with
// SwiGLU the 8 gate rows and the 8 up rows of those columns) over the whole
// k range, so every column is finished in one workgroup (no split-K
// partials) and N = 2048 still spreads over 256 workgroups.  Lane 8r + t
// reads 16 bytes at k = 64c + 8t of row r: each load instruction takes 8
// whole 128-byte lines.  The NW waves take interleaved chunks c, four per
// pass, the next pass's loads in flight while one is summed (a workgroup
// may also walk several tiles in turn; the launch gives each one tile, as
// timing favoured more resident waves over fewer rounds).  The rows of A are
// staged in LDS once per workgroup (zero rows past M), normalised on the way
// when a gain is given:
// one wave per row, sum of squares in lane order, rstd = 1/sqrt(mean + eps),
// A' = bf16(A rstd g), as the row-wise RMSNorm kernel computes it.  Partial
// sums are reduced over the 8 lanes of a row, then over the waves in wave
// order through LDS; the epilogue applies alpha and the residual (and copies
// key/value columns to the cache) or the activation, rounding u and v to
// bf16 first as the unfused path stores them.

constexpr int kDecCols = 8;   // output columns per workgroup
constexpr int kDecU = 4;      // chunks per pass
constexpr int kDecCus = 256;  // compute units

__host__ __device__ inline int dec_pitch(int64_t K) { return static_cast<int>((K + 63) & ~63ll); }

__device__ __forceinline__ float dot8(const bf16x8& w, const bf16x8& a, float c) {
#pragma unroll
  for (int e = 0; e < 8; e += 2)
    c = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{w[e], w[e + 1]}, bf16x2{a[e], a[e + 1]}, c, false);
  return c;
}

template <int NW, int ACT, bool NORM>
__global__ __launch_bounds__(NW * 64) void ld_gemm_bf16_dec(SkinnyArgs g) {
  constexpr int NR = ACT == kDecActSwiglu ? 2 : 1;  // W rows per lane
  extern __shared__ __align__(16) unsigned char dsm[];
  const int M = g.M, N = g.N, K = g.K;
  const int pitch = dec_pitch(K);
  bf16* as = reinterpret_cast<bf16*>(dsm);
  float* red = reinterpret_cast<float*>(dsm + static_cast<size_t>(kDecGemmMaxM) * pitch * 2);
  float* fin = red + NW * NR * kDecCols * kDecGemmMaxM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane >> 3, t = lane & 7;
  const int nchunks = (K + 63) >> 6;
  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* W = static_cast<const bf16*>(g.W);

  // This workgroup's tile: columns col of its lanes' rows; the k range in
  // npass passes of kDecU chunks per wave.
  const int col = blockIdx.x * kDecCols + r;
  const bool nvalid = col < N;
  const int npass = (nchunks + kDecU * NW - 1) / (kDecU * NW);
  const bf16* wrow[NR];
#pragma unroll
  for (int j = 0; j < NR; ++j) wrow[j] = W + static_cast<int64_t>(nvalid ? col + j * N : 0) * g.ldw + 8 * t;

  typedef bf16x8 WBuf[kDecU][NR];
  auto load_w = [&](WBuf& wb, int p) {
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      const int kc = (wave + NW * (kDecU * p + u)) * 64;
#pragma unroll
      for (int j = 0; j < NR; ++j) wb[u][j] = (nvalid && kc + 8 * t < K) ? load8(wrow[j] + kc) : zero8();
    }
  };
  // the first two passes' loads and the epilogue's residual go out before
  // the staging below waits on its own loads
  WBuf w0, w1;
  load_w(w0, 0);
  if (npass > 1) load_w(w1, 1);
  const int em = tid / kDecCols, en = blockIdx.x * kDecCols + tid % kDecCols;  // epilogue element
  const bool eval = tid < M * kDecCols && en < N;
  float resid = 0.f;
  if (ACT == kDecActNone && g.R && eval)
    resid = static_cast<float>(static_cast<const bf16*>(g.R)[static_cast<int64_t>(em) * g.ldr + en]);

  // stage the rows of A (normalised when a gain is given), zero rows past M
  const int k8n = K >> 3, p8 = pitch >> 3;
  for (int m = wave; m < kDecGemmMaxM; m += NW) {
    bf16* dst = as + m * pitch;
    if (m >= M) {
      for (int k8 = lane; k8 < p8; k8 += 64) *reinterpret_cast<bf16x8*>(dst + 8 * k8) = zero8();
      continue;
    }
    const bf16* x = A + static_cast<int64_t>(m) * g.lda;
    if constexpr (NORM) {
      constexpr int NCH = kDecGemmMaxKNorm / 512;
      bf16x8 xv[NCH];
      float ss = 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int k8 = c * 64 + lane;
        if (k8 < k8n) {
          xv[c] = load8(x + 8 * k8);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float f = static_cast<float>(xv[c][e]);
            ss = __builtin_fmaf(f, f, ss);
          }
        }
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
      const float rstd = rsqrtf(ss / static_cast<float>(K) + g.eps);
      const bf16* gain = static_cast<const bf16*>(g.g);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int k8 = c * 64 + lane;
        if (k8 < k8n) {
          const bf16x8 gv = load8(gain + 8 * k8);
          bf16x8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            o[e] = static_cast<bf16>(static_cast<float>(xv[c][e]) * rstd * static_cast<float>(gv[e]));
          *reinterpret_cast<bf16x8*>(dst + 8 * k8) = o;
        }
      }
    } else {
      for (int k8 = lane; k8 < k8n; k8 += 64) *reinterpret_cast<bf16x8*>(dst + 8 * k8) = load8(x + 8 * k8);
    }
    for (int k8 = k8n + lane; k8 < p8; k8 += 64) *reinterpret_cast<bf16x8*>(dst + 8 * k8) = zero8();
  }
  __syncthreads();

  float acc[NR][kDecGemmMaxM];
#pragma unroll
  for (int j = 0; j < NR; ++j)
#pragma unroll
    for (int m = 0; m < kDecGemmMaxM; ++m) acc[j][m] = 0.f;
  auto dots = [&](const WBuf& wb, int p) {
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      const int c = wave + NW * (kDecU * p + u);
      if (c < nchunks) {  // wave-uniform
        const bf16* ak = as + c * 64 + 8 * t;
#pragma unroll
        for (int m = 0; m < kDecGemmMaxM; ++m) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(ak + m * pitch);
#pragma unroll
          for (int j = 0; j < NR; ++j) acc[j][m] = dot8(wb[u][j], a, acc[j][m]);
        }
      }
    }
  };
  for (int p = 0; p < npass; p += 2) {
    dots(w0, p);
    if (p + 2 < npass) load_w(w0, p + 2);
    if (p + 1 < npass) {
      dots(w1, p + 1);
      if (p + 3 < npass) load_w(w1, p + 3);
    }
  }

  // sums over the 8 lanes of a row, then over the waves in wave order
#pragma unroll
  for (int j = 0; j < NR; ++j)
#pragma unroll
    for (int m = 0; m < kDecGemmMaxM; ++m) {
      float v = acc[j][m];
      v += __shfl_xor(v, 1, 8);
      v += __shfl_xor(v, 2, 8);
      v += __shfl_xor(v, 4, 8);
      acc[j][m] = v;
    }
  if (t == 0)
#pragma unroll
    for (int j = 0; j < NR; ++j)
#pragma unroll
      for (int m = 0; m < kDecGemmMaxM; ++m) red[((wave * NR + j) * kDecCols + r) * kDecGemmMaxM + m] = acc[j][m];
  __syncthreads();
  constexpr int kVals = NR * kDecCols * kDecGemmMaxM;
  if (tid < kVals) {
    float sum = 0.f;
    for (int w = 0; w < NW; ++w) sum += red[w * kVals + tid];
    fin[tid] = sum;  // [j][column][row]
  }
  __syncthreads();
  if (eval) {
    const int c = tid % kDecCols;
    bf16* C = static_cast<bf16*>(g.C) + static_cast<int64_t>(em) * g.ldc + en;
    const float s0 = fin[c * kDecGemmMaxM + em];
    if constexpr (ACT == kDecActSwiglu) {
      const float u = bf16r(g.alpha * s0), v = bf16r(g.alpha * fin[(kDecCols + c) * kDecGemmMaxM + em]);
      *C = static_cast<bf16>(swiglu_fwd_f(u, v));
    } else if constexpr (ACT == kDecActRelu2) {
      const float z = fmaxf(bf16r(g.alpha * s0), 0.f);
      *C = static_cast<bf16>(z * z);
    } else {
      const bf16 o = static_cast<bf16>(g.alpha * s0 + resid);
      *C = o;
      if (g.kv && en >= g.kv_d) {
        const int64_t b = em / g.kv_n, jj = em % g.kv_n;
        static_cast<bf16*>(g.kv)[(b * g.kv_s_max + g.kv_pos + jj) * 2 * g.kv_d + (en - g.kv_d)] = o;
      }
    }
  }
}

// ------------------------------------------------------------ KV store

__global__ __launch_bounds__(256) void ld_kv_store_k(KvArgs a) {
  const int64_t per_row = (2ll * a.d) / 8;
  const int64_t total = static_cast<int64_t>(a.n_seq) * a.n * per_row;
  const bf16* src = static_cast<const bf16*>(a.qkv);
  bf16* dst = static_cast<bf16*>(a.cache);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t r = id / per_row, c = (id % per_row) * 8;
    const int64_t b = r / a.n, j = r % a.n;
    const bf16x8 v = load8(src + r * a.ld_qkv + a.d + c);
    *reinterpret_cast<bf16x8*>(dst + ((b * a.s_max + a.pos + j) * 2 * a.d) + c) = v;
  }
}

// ------------------------------------------------------ decode attention

// NQ >= n_new query rows per sequence (1, 2, 4 or 8).  A wave covers 64 keys
// of the chunk: DH/8 lanes per key row, 8 dimensions (16 bytes) each, so a
// pass covers 64/(DH/8) keys and all passes' loads are issued before any
// arithmetic.
template <int DH, int NQ>
__global__ __launch_bounds__(256) void ld_attn_decode_bf16(DecAttnArgs a) {
  constexpr int LPK = DH / 8;    // lanes per key row
  constexpr int KPP = 64 / LPK;  // keys per pass
  constexpr int NP = 64 / KPP;   // passes per wave
  __shared__ float sc[NQ][kDecKeys + 1];  // + 1: the MFMA path's rows in different banks
  __shared__ float red[4][NQ][DH];
  const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = lane / LPK, sl = lane % LPK;
  const int d = a.H * DH;
  const int64_t row2 = 2ll * d;
  const int nk = a.pos + a.n_new;
  const int k0 = c * kDecKeys + wave * 64;
  const float al2 = a.alibi ? alibi_slope(h, a.H) * kLog2e : 0.f;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* cache = static_cast<const bf16*>(a.cache) + static_cast<int64_t>(b) * a.s_max * row2;

  if constexpr (NQ == 1) {
    // one query row: each lane's 8 dimensions of a key, dot products summed
    // over the key's lanes (keys of rows past the last position read row 0)
    bf16x8 kr[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int kk = k0 + p * KPP + kg;
      kr[p] = load8(cache + static_cast<int64_t>(kk < nk ? kk : 0) * row2 + h * DH + sl * 8);
    }
    float q[8];
    {
      const bf16x8 v = load8(qkv + static_cast<int64_t>(b) * a.ld_qkv + h * DH + sl * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) q[e] = static_cast<float>(v[e]) * (a.scale * kLog2e);
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int kl = wave * 64 + p * KPP + kg;
      const int kk = k0 + p * KPP + kg;
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s = __builtin_fmaf(q[e], static_cast<float>(kr[p][e]), s);
#pragma unroll
      for (int o = LPK / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
      if (sl == 0) sc[0][kl] = (kk < nk && kk <= a.pos) ? s - al2 * static_cast<float>(a.pos - kk) : -INFINITY;
    }
  } else {
    // several query rows: S^T = K Q^T on the matrix cores, the wave's 64 keys
    // in two 32-key blocks (A operand: lane l holds key l % 32, dimensions
    // 16 ks + 8 (l / 32) .. +7), the query rows as the 32 columns (B operand;
    // rows past n_new are zero).  Lane l, register v of block kb then holds
    // key 32 kb + 8 (v / 4) + 4 (l / 32) + v % 4 of query row l % 32.
    const int ql = lane & 31, hf = lane >> 5;
    bf16x8 qf[DH / 16], kf[2][DH / 16];
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks)
      qf[ks] = ql < a.n_new ? load8(qkv + (static_cast<int64_t>(b) * a.n_new + ql) * a.ld_qkv + h * DH + 16 * ks + 8 * hf)
                            : zero8();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int kk = k0 + kb * 32 + ql;
      const bf16* kp = cache + static_cast<int64_t>(kk < nk ? kk : 0) * row2 + h * DH + 8 * hf;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) kf[kb][ks] = load8(kp + 16 * ks);
    }
    floatx16 acc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[kb][v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks)
        acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kb][ks], qf[ks], acc[kb], 0, 0, 0);
    }
    if (ql < a.n_new) {
      const int qpos = a.pos + ql;
      const float sl2 = a.scale * kLog2e;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kl = 32 * kb + 8 * (v >> 2) + 4 * hf + (v & 3);
          const int kk = k0 + kl;
          sc[ql][wave * 64 + kl] =
              (kk < nk && kk <= qpos) ? acc[kb][v] * sl2 - al2 * static_cast<float>(qpos - kk) : -INFINITY;
        }
    }
  }
  // values of the same positions, in flight during the softmax
  bf16x8 vr[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int kk = k0 + p * KPP + kg;
    vr[p] = load8(cache + static_cast<int64_t>(kk < nk ? kk : 0) * row2 + d + h * DH + sl * 8);
  }
  __syncthreads();

  // per query row: chunk maximum, probabilities, sum
  const int64_t prow = (static_cast<int64_t>(b) * a.H + h) * a.n_chunks + c;
  for (int j = wave; j < a.n_new; j += 4) {
    float m = -INFINITY;
    for (int i = lane; i < kDecKeys; i += 64) m = fmaxf(m, sc[j][i]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float l = 0.f;
    for (int i = lane; i < kDecKeys; i += 64) {
      const float pr = m == -INFINITY ? 0.f : exp2f(sc[j][i] - m);
      sc[j][i] = pr;
      l += pr;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o, 64);
    if (lane == 0) {
      a.part_ml[(prow * kDecMaxRows + j) * 2] = m;
      a.part_ml[(prow * kDecMaxRows + j) * 2 + 1] = l;
    }
  }
  __syncthreads();

  // P V in groups of at most four rows: each lane its key's 8 dimensions,
  // then a sum over the wave's key groups (lane exchanges) and over the four
  // waves (LDS, in wave order)
  constexpr int JG = NQ < 4 ? NQ : 4;
#pragma unroll 1
  for (int j0 = 0; j0 < NQ; j0 += JG) {
    float o[JG][8];
#pragma unroll
    for (int j = 0; j < JG; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[j][e] = 0.f;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int kl = wave * 64 + p * KPP + kg;
#pragma unroll
      for (int j = 0; j < JG; ++j) {
        const float pr = j0 + j < a.n_new ? sc[j0 + j][kl] : 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[j][e] = __builtin_fmaf(pr, static_cast<float>(vr[p][e]), o[j][e]);
      }
    }
#pragma unroll
    for (int j = 0; j < JG; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int off = LPK; off < 64; off <<= 1) o[j][e] += __shfl_xor(o[j][e], off, 64);
    if (kg == 0)
#pragma unroll
      for (int j = 0; j < JG; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) red[wave][j0 + j][sl * 8 + e] = o[j][e];
  }
  __syncthreads();
  for (int e = tid; e < a.n_new * DH; e += 256) {
    const int j = e / DH, col = e % DH;
    const float s = red[0][j][col] + red[1][j][col] + red[2][j][col] + red[3][j][col];
    a.part_o[(prow * kDecMaxRows + j) * DH + col] = s;
  }
}

// One wave per (sequence, head, query row): merge the chunks.
template <int DH>
__global__ __launch_bounds__(256) void ld_attn_decode_combine(DecAttnArgs a) {
  constexpr int NQ = kDecMaxRows;   // row stride of the partials
  constexpr int CL = DH / 64;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= a.n_seq * a.H * a.n_new) return;
  const int b = r / (a.H * a.n_new), h = (r / a.n_new) % a.H, j = r % a.n_new;
  const int64_t p0 = (static_cast<int64_t>(b) * a.H + h) * a.n_chunks;
  float M = -INFINITY;
  for (int c = 0; c < a.n_chunks; ++c) M = fmaxf(M, a.part_ml[((p0 + c) * NQ + j) * 2]);
  float L = 0.f, acc[CL];
#pragma unroll
  for (int cc = 0; cc < CL; ++cc) acc[cc] = 0.f;
  for (int c = 0; c < a.n_chunks; ++c) {
    const float mc = a.part_ml[((p0 + c) * NQ + j) * 2];
    const float wgt = mc == -INFINITY ? 0.f : exp2f(mc - M);
    L = __builtin_fmaf(wgt, a.part_ml[((p0 + c) * NQ + j) * 2 + 1], L);
#pragma unroll
    for (int cc = 0; cc < CL; ++cc)
      acc[cc] = __builtin_fmaf(wgt, a.part_o[((p0 + c) * NQ + j) * DH + lane * CL + cc], acc[cc]);
  }
  const float inv = 1.f / L;
  bf16* out = static_cast<bf16*>(a.out) + (static_cast<int64_t>(b) * a.n_new + j) * (a.H * DH) + h * DH;
#pragma unroll
  for (int cc = 0; cc < CL; ++cc) out[lane * CL + cc] = static_cast<bf16>(acc[cc] * inv);
}

int grid_for(int64_t items) {
  int64_t g = (items + 255) / 256;
  if (g > 8192) g = 8192;
  if (g < 1) g = 1;
  return static_cast<int>(g);
}

}  // namespace

int skinny_ksplit(int64_t M, int64_t N, int64_t K) {
  (void)M;
  const int64_t tiles = (N + 31) / 32;
  const int64_t chunks = (K + kSkChunk - 1) / kSkChunk;
  int64_t ks = (512 + tiles - 1) / tiles;
  const int64_t most = chunks / kSkWaves;
  if (ks > most) ks = most;
  if (ks > 16) ks = 16;
  if (ks < 1) ks = 1;
  return static_cast<int>(ks);
}

hipError_t launch_gemm_skinny(const SkinnyArgs& g, int ksplit, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const dim3 grid((g.N + 31) / 32, ksplit);
  if (g.M <= 32)
    hipLaunchKernelGGL(ld_gemm_bf16_skinny<1>, grid, dim3(256), 0, s, g);
  else
    hipLaunchKernelGGL(ld_gemm_bf16_skinny<2>, grid, dim3(256), 0, s, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ksplit == 1 || g.part_only) return e;
  hipLaunchKernelGGL(ld_skinny_reduce_k, dim3(grid_for(static_cast<int64_t>(g.M) * g.N)), dim3(256), 0,
                     s, g, ksplit);
  return hipGetLastError();
}

size_t dec_gemm_lds_bytes(int64_t K, int nw) {
  return static_cast<size_t>(kDecGemmMaxM) * dec_pitch(K) * 2 +
         static_cast<size_t>(nw + 1) * 2 * kDecCols * kDecGemmMaxM * 4;
}

bool dec_gemm_ok(int64_t M, int64_t K, bool norm) {
  return M >= 1 && M <= kDecGemmMaxM && K >= 8 && K % 8 == 0 && (!norm || K <= kDecGemmMaxKNorm) &&
         dec_gemm_lds_bytes(K, 16) <= 160 * 1024;
}

template <int NW, int ACT>
hipError_t gemm_dec_t(const SkinnyArgs& g, int tiles, hipStream_t s) {
  const size_t lds = dec_gemm_lds_bytes(g.K, NW);
  if (g.g)
    hipLaunchKernelGGL((ld_gemm_bf16_dec<NW, ACT, true>), dim3(tiles), dim3(NW * 64), lds, s, g);
  else
    hipLaunchKernelGGL((ld_gemm_bf16_dec<NW, ACT, false>), dim3(tiles), dim3(NW * 64), lds, s, g);
  return hipGetLastError();
}

hipError_t launch_gemm_dec(const SkinnyArgs& g, hipStream_t s) {
  if (g.N <= 0) return hipSuccess;
  if (!dec_gemm_ok(g.M, g.K, g.g != nullptr)) return hipErrorInvalidValue;
  const int tiles = (g.N + kDecCols - 1) / kDecCols;
  // One workgroup per tile, all resident at once: while the tiles fit one
  // per CU, 16 waves (8 with SwiGLU, whose two rows per lane need more than
  // the 128 registers of 16 waves), else 4 (up to four workgroups per CU);
  // either way every wave's loads are issued up front.
  if (g.act == kDecActSwiglu)
    return tiles <= kDecCus ? gemm_dec_t<8, kDecActSwiglu>(g, tiles, s) : gemm_dec_t<4, kDecActSwiglu>(g, tiles, s);
  if (g.act == kDecActRelu2)
    return tiles <= kDecCus ? gemm_dec_t<16, kDecActRelu2>(g, tiles, s) : gemm_dec_t<4, kDecActRelu2>(g, tiles, s);
  return tiles <= kDecCus ? gemm_dec_t<16, kDecActNone>(g, tiles, s) : gemm_dec_t<4, kDecActNone>(g, tiles, s);
}

hipError_t launch_skinny_reduce_norm(const SkinnyArgs& g, int ksplit, const void* gain, float eps, void* h,
                                     hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  hipLaunchKernelGGL(ld_skinny_reduce_norm_k, dim3(g.M), dim3(1024), 0, s, g, ksplit, static_cast<const bf16*>(gain),
                     eps, static_cast<bf16*>(h));
  return hipGetLastError();
}

hipError_t launch_skinny_reduce_act(const SkinnyArgs& g, int ksplit, int act, int f, void* s_out, hipStream_t s) {
  if (g.M <= 0 || f <= 0) return hipSuccess;
  hipLaunchKernelGGL(ld_skinny_reduce_act_k, dim3(grid_for(static_cast<int64_t>(g.M) * f)), dim3(256), 0, s, g,
                     ksplit, act, f, static_cast<bf16*>(s_out));
  return hipGetLastError();
}

hipError_t launch_kv_store(const KvArgs& a, hipStream_t s) {
  const int64_t items = static_cast<int64_t>(a.n_seq) * a.n * (2ll * a.d / 8);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(ld_kv_store_k, dim3(grid_for(items)), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int DH, int NQ>
hipError_t attn_decode_t(const DecAttnArgs& a, hipStream_t s) {
  const dim3 grid(a.n_chunks, a.H, a.n_seq);
  hipLaunchKernelGGL((ld_attn_decode_bf16<DH, NQ>), grid, dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows = a.n_seq * a.H * a.n_new;
  hipLaunchKernelGGL(ld_attn_decode_combine<DH>, dim3((rows + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int DH>
hipError_t attn_decode_dh(const DecAttnArgs& a, hipStream_t s) {
  if (a.n_new <= 1) return attn_decode_t<DH, 1>(a, s);
  if (a.n_new <= 2) return attn_decode_t<DH, 2>(a, s);
  if (a.n_new <= 4) return attn_decode_t<DH, 4>(a, s);
  return attn_decode_t<DH, 8>(a, s);
}

hipError_t launch_attn_decode(const DecAttnArgs& a, hipStream_t s) {
  return a.dh == 128 ? attn_decode_dh<128>(a, s) : attn_decode_dh<64>(a, s);
}

}  // namespace ld

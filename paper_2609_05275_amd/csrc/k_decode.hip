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
// second kernel, so results do not depend on timing.
//
// Decode attention: one workgroup per (256-key chunk, head, sequence).
// Scores: eight lanes per key, each holding an eighth of the head's
// dimensions of every query row, reduced by three lane exchanges; scores in
// base 2 with the causal cut (key <= query position) and the ALiBi bias.
// Softmax statistics per query row over the chunk, then P V with a lane per
// head dimension (coalesced value reads), the four waves' key ranges summed
// in LDS.  A combine kernel merges the chunks with the usual max/sum
// rescaling and writes bf16.
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
  static_cast<bf16*>(g.C)[static_cast<int64_t>(m) * g.ldc + n] = static_cast<bf16>(v);
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

  for (int c = blockIdx.y * kSkWaves + wave; c < nchunks; c += workers) {
    const int kc = c * kSkChunk;
    bf16x8 b[4], a[MB][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bool kv = kc + 32 * h + 8 * s < g.K;   // K % 8 == 0: the whole 8 are in range
      b[s] = (nvalid && kv) ? load8(wrow + kc + 8 * s) : zero8();
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        a[mb][s] = (mvalid[mb] && kv) ? load8(arow[mb] + kc + 8 * s) : zero8();
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mb][s], b[s], acc[mb], 0, 0, 0);
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
      if (gridDim.y > 1)
        g.part[(static_cast<int64_t>(blockIdx.y) * g.M + m) * g.N + n] = sum;
      else
        skinny_store(g, m, n, sum);
    }
  }
}

__global__ __launch_bounds__(256) void ld_skinny_reduce_k(SkinnyArgs g, int ksplit) {
  const int64_t total = static_cast<int64_t>(g.M) * g.N;
  const int64_t plane = total;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < total; i += gridDim.x * 256ll) {
    float sum = g.part[i];
    for (int s = 1; s < ksplit; ++s) sum += g.part[s * plane + i];
    skinny_store(g, static_cast<int>(i / g.N), static_cast<int>(i % g.N), sum);
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

template <int DH>
__global__ __launch_bounds__(256) void ld_attn_decode_bf16(DecAttnArgs a) {
  constexpr int NQ = kDecMaxRows;
  constexpr int EL = DH / 8;   // dimensions per lane of a key row
  constexpr int CL = DH / 64;  // value columns per lane
  __shared__ float sc[NQ][kDecKeys];
  __shared__ float red[4][NQ][DH];
  const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.H * DH;
  const int64_t row2 = 2ll * d;
  const int nk = a.pos + a.n_new;
  const int k0 = c * kDecKeys;
  const float al2 = a.alibi ? alibi_slope(h, a.H) * kLog2e : 0.f;
  const int grp = lane >> 3, sl = lane & 7;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* cache = static_cast<const bf16*>(a.cache) + static_cast<int64_t>(b) * a.s_max * row2;

  float q[NQ][EL];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const bool jv = j < a.n_new;
    const bf16* qp = qkv + (static_cast<int64_t>(b) * a.n_new + (jv ? j : 0)) * a.ld_qkv + h * DH + sl * EL;
#pragma unroll
    for (int e8 = 0; e8 < EL / 8; ++e8) {
      const bf16x8 v = jv ? load8(qp + 8 * e8) : zero8();
#pragma unroll
      for (int e = 0; e < 8; ++e) q[j][8 * e8 + e] = static_cast<float>(v[e]) * (a.scale * kLog2e);
    }
  }

  // scores: each wave 64 keys of the chunk, 8 keys per pass
  const bf16* kbase = cache + h * DH + sl * EL;
  for (int it = 0; it < 8; ++it) {
    const int kl = wave * 64 + it * 8 + grp;
    const int kk = k0 + kl;
    const bool valid = kk < nk;
    float kv[EL];
#pragma unroll
    for (int e8 = 0; e8 < EL / 8; ++e8) {
      const bf16x8 v = load8(kbase + static_cast<int64_t>(valid ? kk : 0) * row2 + 8 * e8);
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[8 * e8 + e] = static_cast<float>(v[e]);
    }
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      if (j < a.n_new) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < EL; ++e) s = __builtin_fmaf(q[j][e], kv[e], s);
        s += __shfl_xor(s, 1, 64);
        s += __shfl_xor(s, 2, 64);
        s += __shfl_xor(s, 4, 64);
        const int qpos = a.pos + j;
        if (sl == 0)
          sc[j][kl] = (valid && kk <= qpos) ? s - al2 * static_cast<float>(qpos - kk) : -INFINITY;
      }
    }
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
      const float p = m == -INFINITY ? 0.f : exp2f(sc[j][i] - m);
      sc[j][i] = p;
      l += p;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o, 64);
    if (lane == 0) {
      a.part_ml[(prow * NQ + j) * 2] = m;
      a.part_ml[(prow * NQ + j) * 2 + 1] = l;
    }
  }
  __syncthreads();

  // P V over this wave's 64 keys
  float o[NQ][CL];
#pragma unroll
  for (int j = 0; j < NQ; ++j)
#pragma unroll
    for (int cc = 0; cc < CL; ++cc) o[j][cc] = 0.f;
  int kn = nk - (k0 + wave * 64);
  kn = kn < 0 ? 0 : (kn > 64 ? 64 : kn);
  const bf16* vbase = cache + d + h * DH + lane * CL;
#pragma unroll 4
  for (int i = 0; i < kn; ++i) {
    const int kl = wave * 64 + i;
    const bf16* vp = vbase + static_cast<int64_t>(k0 + kl) * row2;
    float v[CL];
    if constexpr (CL == 2) {
      const bf16x2 pr = *reinterpret_cast<const bf16x2*>(vp);
      v[0] = static_cast<float>(pr[0]);
      v[1] = static_cast<float>(pr[CL - 1]);
    } else {
      v[0] = static_cast<float>(vp[0]);
    }
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      if (j < a.n_new) {
        const float p = sc[j][kl];
#pragma unroll
        for (int cc = 0; cc < CL; ++cc) o[j][cc] = __builtin_fmaf(p, v[cc], o[j][cc]);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NQ; ++j)
    if (j < a.n_new)
#pragma unroll
      for (int cc = 0; cc < CL; ++cc) red[wave][j][lane * CL + cc] = o[j][cc];
  __syncthreads();
  for (int e = tid; e < a.n_new * DH; e += 256) {
    const int j = e / DH, col = e % DH;
    const float s = red[0][j][col] + red[1][j][col] + red[2][j][col] + red[3][j][col];
    a.part_o[(prow * NQ + j) * DH + col] = s;
  }
}

// One wave per (sequence, head, query row): merge the chunks.
template <int DH>
__global__ __launch_bounds__(256) void ld_attn_decode_combine(DecAttnArgs a) {
  constexpr int NQ = kDecMaxRows;
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
  if (e != hipSuccess || ksplit == 1) return e;
  hipLaunchKernelGGL(ld_skinny_reduce_k, dim3(grid_for(static_cast<int64_t>(g.M) * g.N)), dim3(256), 0,
                     s, g, ksplit);
  return hipGetLastError();
}

hipError_t launch_kv_store(const KvArgs& a, hipStream_t s) {
  const int64_t items = static_cast<int64_t>(a.n_seq) * a.n * (2ll * a.d / 8);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(ld_kv_store_k, dim3(grid_for(items)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_decode(const DecAttnArgs& a, hipStream_t s) {
  const dim3 grid(a.n_chunks, a.H, a.n_seq);
  const int rows = a.n_seq * a.H * a.n_new;
  const dim3 cgrid((rows + 3) / 4);
  if (a.dh == 128) {
    hipLaunchKernelGGL(ld_attn_decode_bf16<128>, grid, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ld_attn_decode_combine<128>, cgrid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(ld_attn_decode_bf16<64>, grid, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ld_attn_decode_combine<64>, cgrid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ld

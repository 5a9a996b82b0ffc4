// Mask + compaction, row gather / scatter-add, RMSNorm and SwiGLU kernels.
// All of these are HBM-bound: 16-byte vector accesses, one wave per row for
// the normalisations, fp32 arithmetic on bf16 or fp32 storage.
#include <type_traits>

#include "ld_internal.h"

namespace ld {
namespace {

// ------------------------------------------------------------ utilities

template <typename T>
struct alignas(16) Pack {
  static constexpr int N = 16 / sizeof(T);
  T v[N];
};

template <typename T>
__device__ __forceinline__ Pack<T> load16(const T* p) {
  return *reinterpret_cast<const Pack<T>*>(p);
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const Pack<T>& v) {
  *reinterpret_cast<Pack<T>*>(p) = v;
}

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16 x) { return static_cast<float>(x); }
template <typename T>
__device__ __forceinline__ T from_f(float x) {
  return static_cast<T>(x);  // round to nearest even (v_cvt_pk_bf16_f32 for bf16)
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int64_t row_count(const RowCount& rc) {
  return rc.dev_count ? static_cast<int64_t>(*rc.dev_count) * rc.mult : rc.rows;
}

__device__ __forceinline__ int64_t map_row(const RowMap& m, int64_t row) {
  if (!m.idx) return row;
  return static_cast<int64_t>(m.idx[row / m.S]) * m.S + row % m.S;
}

// ------------------------------------------------------------- masks

// One workgroup per (layer, mask).  Each chunk of blockDim samples draws its bits,
// a 64-wide ballot + popcount of the lower lanes gives each kept sample its
// rank inside the wave, and a serial scan of the per-wave totals in LDS gives
// the wave offsets, so the kept list comes out ascending.
__global__ __launch_bounds__(1024) void ld_mask_compact(MaskArgs a) {
  __shared__ int wave_tot[16];
  const int layer = blockIdx.x / a.n_masks, m = blockIdx.x % a.n_masks;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_waves = blockDim.x >> 6;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * a.batch;
  int base = 0;
  for (int b0 = 0; b0 < a.batch; b0 += blockDim.x) {
    const int b = b0 + tid;
    int keep = 0;
    if (b < a.batch) {
      if (a.keep_override) {
        keep = a.keep_override[row + b] != 0;
      } else if (!a.drop_all[layer]) {
        const uint64_t w = mask_draw(static_cast<uint64_t>(b),
                                     static_cast<uint64_t>(a.first_layer + layer), a.step, a.seed,
                                     a.per_batch, m);
        keep = !(w < a.thr[layer]);
      }
      a.keep[row + b] = static_cast<uint8_t>(keep);
    }
    const uint64_t ball = __ballot(keep);
    const int rank = __popcll(ball & ((1ull << lane) - 1ull));
    if (lane == 0) wave_tot[wave] = __popcll(ball);
    __syncthreads();
    int off = base, tot = 0;
    for (int w = 0; w < n_waves; ++w) {
      if (w < wave) off += wave_tot[w];
      tot += wave_tot[w];
    }
    if (keep) a.idx[row + off + rank] = b;
    __syncthreads();
    base += tot;
  }
  for (int j = base + tid; j < a.batch; j += blockDim.x) a.idx[row + j] = -1;
  if (tid == 0) {
    a.count[blockIdx.x] = base;
    if (a.r_out && m == 0) a.r_out[layer] = a.r[layer];
  }
}

__global__ __launch_bounds__(256) void ld_zero_f32_k(ZeroArgs a) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int i = 0; i < a.count; ++i) {
    float* p = a.p[i];
    const int64_t n = a.n[i];
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const int64_t n4 = n / 4;
      for (int64_t j = t0; j < n4; j += stride) reinterpret_cast<float4*>(p)[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int64_t j = n4 * 4 + t0; j < n; j += stride) p[j] = 0.f;
    } else {
      for (int64_t j = t0; j < n; j += stride) p[j] = 0.f;
    }
  }
}

// ------------------------------------------------------- gather / scatter

// Chunks of VN consecutive elements (8 or 16, 16 or 32 bytes per lane).
template <typename T, int VN>
struct alignas(sizeof(T) * VN < 16 ? sizeof(T) * VN : 16) Chunk {
  T v[VN];
};
template <typename T, int VN>
__device__ __forceinline__ Chunk<T, VN> ldc(const T* p) {
  return *reinterpret_cast<const Chunk<T, VN>*>(p);
}
template <typename T, int VN>
__device__ __forceinline__ void stc(T* p, const Chunk<T, VN>& c) {
  *reinterpret_cast<Chunk<T, VN>*>(p) = c;
}

// Row gather: dst rows (type TD) from src rows (type TS) through the row
// maps; a bit copy when the types agree, one rounding to nearest even when
// float32 rows go to bf16.
template <typename TS, typename TD>
__global__ __launch_bounds__(256) void ld_gather_rows_k(RowsArgs a) {
  constexpr int VN = 16 / sizeof(TD);
  const int64_t chunks = a.d / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const TS* src = static_cast<const TS*>(a.src);
  TD* dst = static_cast<TD*>(a.dst);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    const Chunk<TS, VN> v = ldc<TS, VN>(src + map_row(a.src_map, row) * a.d + c);
    if constexpr (std::is_same<TS, TD>::value) {
      stc<TD, VN>(dst + map_row(a.dst_map, row) * a.d + c, v);
    } else {
      Chunk<TD, VN> o;
#pragma unroll
      for (int i = 0; i < VN; ++i) o.v[i] = from_f<TD>(to_f(v.v[i]));
      stc<TD, VN>(dst + map_row(a.dst_map, row) * a.d + c, o);
    }
  }
}

// bf16 <-> float32 over n elements (8 per thread and step).
template <typename TS, typename TD>
__global__ __launch_bounds__(256) void ld_convert_k(const TS* src, TD* dst, int64_t n8) {
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < n8; id += gridDim.x * 256ll) {
    const Chunk<TS, 8> v = ldc<TS, 8>(src + id * 8);
    Chunk<TD, 8> o;
#pragma unroll
    for (int i = 0; i < 8; ++i) o.v[i] = from_f<TD>(to_f(v.v[i]));
    stc<TD, 8>(dst + id * 8, o);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void ld_scatter_add_rows_k(RowsArgs a) {
  constexpr int VN = Pack<T>::N;
  const int64_t chunks = a.d / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const T* y = static_cast<const T*>(a.src);
  T* x = static_cast<T*>(a.dst);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    T* xp = x + map_row(a.dst_map, row) * a.d + c;
    const Pack<T> yv = load16(y + map_row(a.src_map, row) * a.d + c);
    Pack<T> xv = load16(xp);
#pragma unroll
    for (int i = 0; i < VN; ++i) xv.v[i] = from_f<T>(__builtin_fmaf(a.r, to_f(yv.v[i]), to_f(xv.v[i])));
    store16(xp, xv);
  }
}

// ---------------------------------------------------------------- RMSNorm
// One wave per row; a lane holds NCH chunks of VN consecutive elements (VN =
// 8 in bf16 configurations, 4 in float32 ones).  Each tensor has its own
// element type (see RmsFwdArgs / RmsBwdArgs): the source rows of the forward
// and the saved inputs, residual gradients and outputs of the backward may be
// float32 (the residual streams) while the GEMM operands are bf16.

template <typename TS, typename TY, int VN, int NCH>
__global__ __launch_bounds__(256) void ld_rmsnorm_fwd_k(RmsFwdArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = blockIdx.x * 4ll + wave;
  if (row >= row_count(a.rc)) return;
  const TS* x = static_cast<const TS*>(a.x) + map_row(a.src, row) * a.d;
  const TY* g = static_cast<const TY*>(a.g);
  Chunk<TS, VN> v[NCH];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = (c * 64 + lane) * VN;
    if (col < a.d) {
      v[c] = ldc<TS, VN>(x + col);
#pragma unroll
      for (int i = 0; i < VN; ++i) {
        const float f = to_f(v[c].v[i]);
        ss = __builtin_fmaf(f, f, ss);
      }
    }
  }
  ss = wave_sum(ss);
  const float rstd = rsqrtf(ss / static_cast<float>(a.d) + a.eps);
  TY* y = static_cast<TY*>(a.y) + row * a.d;
  float* xc = a.xcopy ? a.xcopy + row * a.d : nullptr;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = (c * 64 + lane) * VN;
    if (col < a.d) {
      if (xc) {
        Chunk<float, VN> cc;
#pragma unroll
        for (int i = 0; i < VN; ++i) cc.v[i] = to_f(v[c].v[i]);
        stc<float, VN>(xc + col, cc);
      }
      const Chunk<TY, VN> gv = ldc<TY, VN>(g + col);
      Chunk<TY, VN> o;
#pragma unroll
      for (int i = 0; i < VN; ++i) o.v[i] = from_f<TY>(to_f(v[c].v[i]) * rstd * to_f(gv.v[i]));
      stc<TY, VN>(y + col, o);
    }
  }
  if (lane == 0) a.rstd[row] = rstd;
}

constexpr int kBwdRowsPerBlock = 16;

template <typename TX, typename TY, typename TR, int VN, int NCH>
struct NormRow {
  Chunk<TX, VN> x[NCH];
  Chunk<TY, VN> gy[NCH];
  Chunk<TR, VN> res[NCH];
  float rstd;
};

// Column of chunk c of thread t: (c * 256 + t) * VN.
template <typename TX, typename TY, typename TR, int VN, int NCH>
__device__ __forceinline__ void norm_row_load(NormRow<TX, TY, TR, VN, NCH>& r, const RmsBwdArgs& a, int64_t row,
                                              int tid) {
  const TX* x = static_cast<const TX*>(a.x) + row * a.d;
  const TY* gy = static_cast<const TY*>(a.gy) + row * a.d;
  const TR* gres = a.gres ? static_cast<const TR*>(a.gres) + map_row(a.res_map, row) * a.d : nullptr;
  r.rstd = a.rstd[row];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = (c * 256 + tid) * VN;
    if (col < a.d) {
      r.x[c] = ldc<TX, VN>(x + col);
      r.gy[c] = ldc<TY, VN>(gy + col);
      if (gres) r.res[c] = ldc<TR, VN>(gres + col);
    }
  }
}

// gx = gres + rstd*(g*gy) - x*rstd^3*mean_d(x*g*gy), written through the dst
// map (type TO) and, when gx2 is set, as a compacted copy in the
// configuration's type.  A workgroup takes a strip of kBwdRowsPerBlock rows;
// thread t owns the same columns of every row, so its dg = sum_rows gy*x*rstd
// is summed in registers (rows in order) and written as the block's partial
// with no cross-thread reduction.  A row's dot product is summed over the
// wave (shuffles), then over the 4 waves in order through LDS (two slots by
// row parity: one barrier per row).  The next row's loads are issued before
// the current row's reduction.
template <typename TX, typename TY, typename TR, typename TO, int VN, int NCH>
__global__ __launch_bounds__(256) void ld_rmsnorm_bwd_k(RmsBwdArgs a) {
  __shared__ float red[2][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t rows = row_count(a.rc);
  const int64_t r0 = blockIdx.x * static_cast<int64_t>(kBwdRowsPerBlock);
  const int64_t r1 = min(r0 + kBwdRowsPerBlock, rows);
  const TY* gp = static_cast<const TY*>(a.g);
  Chunk<TY, VN> graw[NCH];
  float dga[NCH][VN];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = (c * 256 + tid) * VN;
    if (col < a.d) {
      graw[c] = ldc<TY, VN>(gp + col);
    } else {
#pragma unroll
      for (int i = 0; i < VN; ++i) graw[c].v[i] = from_f<TY>(0.f);
    }
#pragma unroll
    for (int i = 0; i < VN; ++i) dga[c][i] = 0.f;
  }
  const float inv_d = 1.f / static_cast<float>(a.d);
  NormRow<TX, TY, TR, VN, NCH> cur, nxt;
  if (r0 < r1) norm_row_load(cur, a, r0, tid);
  for (int64_t row = r0; row < r1; ++row) {
    if (row + 1 < r1) norm_row_load(nxt, a, row + 1, tid);
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int col = (c * 256 + tid) * VN;
      if (col < a.d) {
#pragma unroll
        for (int i = 0; i < VN; ++i)
          dot = __builtin_fmaf(to_f(cur.x[c].v[i]) * to_f(graw[c].v[i]), to_f(cur.gy[c].v[i]), dot);
      }
    }
    dot = wave_sum(dot);
    const int slot = static_cast<int>(row - r0) & 1;
    if (lane == 0) red[slot][wave] = dot;
    __syncthreads();
    dot = ((red[slot][0] + red[slot][1]) + red[slot][2]) + red[slot][3];
    const float rstd = cur.rstd;
    const float coef = rstd * rstd * rstd * dot * inv_d;
    TO* gx = static_cast<TO*>(a.gx) + map_row(a.dst, row) * a.d;
    TY* gx2 = a.gx2 ? static_cast<TY*>(a.gx2) + row * a.d : nullptr;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int col = (c * 256 + tid) * VN;
      if (col < a.d) {
        Chunk<TO, VN> o;
        Chunk<TY, VN> o2;
#pragma unroll
        for (int i = 0; i < VN; ++i) {
          const float xf = to_f(cur.x[c].v[i]), gyf = to_f(cur.gy[c].v[i]);
          float val = rstd * to_f(graw[c].v[i]) * gyf - xf * coef;
          if (a.gres) val += to_f(cur.res[c].v[i]);
          o.v[i] = from_f<TO>(val);
          o2.v[i] = from_f<TY>(val);
          dga[c][i] = __builtin_fmaf(gyf * xf, rstd, dga[c][i]);
        }
        stc<TO, VN>(gx + col, o);
        if (gx2) stc<TY, VN>(gx2 + col, o2);
      }
    }
    cur = nxt;
  }
  float* part = a.dg_part + static_cast<int64_t>(blockIdx.x) * a.d;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = (c * 256 + tid) * VN;
    if (col < a.d) {
      Chunk<float, VN> o;
#pragma unroll
      for (int i = 0; i < VN; ++i) o.v[i] = dga[c][i];
      stc<float, VN>(part + col, o);
    }
  }
}

// dg[c] = sum over blocks of part[b][c] in a fixed order: 32 row-strided
// partial sums per column (b = r, r+32, ...), then those 32 in order.  A
// workgroup covers 32 columns with 32 row groups, so the d / 32 workgroups
// keep many loads in flight.
constexpr int kDgCols = 32, kDgGroups = 32;
__global__ __launch_bounds__(1024) void ld_dg_reduce_k(const float* part, int64_t n_blocks, int d,
                                                       float* dg) {
  __shared__ float acc[kDgGroups][kDgCols + 1];
  const int c = threadIdx.x % kDgCols, r = threadIdx.x / kDgCols;
  const int col = blockIdx.x * kDgCols + c;
  float sum = 0.f;
  if (col < d) {
    int64_t b = r;
    for (; b + 3 * kDgGroups < n_blocks; b += 4 * kDgGroups) {
      const float v0 = part[b * d + col], v1 = part[(b + kDgGroups) * d + col];
      const float v2 = part[(b + 2 * kDgGroups) * d + col], v3 = part[(b + 3 * kDgGroups) * d + col];
      sum = (((sum + v0) + v1) + v2) + v3;
    }
    for (; b < n_blocks; b += kDgGroups) sum += part[b * d + col];
  }
  acc[r][c] = sum;
  __syncthreads();
  if (r == 0 && col < d) {
    float t = 0.f;
    for (int k = 0; k < kDgGroups; ++k) t += acc[k][c];
    dg[col] = t;
  }
}

// ----------------------------------------------------------------- SwiGLU

template <typename T>
__global__ __launch_bounds__(256) void ld_swiglu_fwd_k(EltArgs a) {
  constexpr int VN = Pack<T>::N;
  const int64_t chunks = a.f / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const T* uv = static_cast<const T*>(a.a);
  T* s = static_cast<T*>(a.out);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    const Pack<T> u = load16(uv + row * 2 * a.f + c);
    const Pack<T> v = load16(uv + row * 2 * a.f + a.f + c);
    Pack<T> o;
#pragma unroll
    for (int i = 0; i < VN; ++i) {
      const float uf = to_f(u.v[i]);
      o.v[i] = from_f<T>(swiglu_fwd_f(uf, to_f(v.v[i])));
    }
    store16(s + row * a.f + c, o);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void ld_swiglu_bwd_k(EltArgs a) {
  constexpr int VN = Pack<T>::N;
  const int64_t chunks = a.f / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const T* uv = static_cast<const T*>(a.a);
  const T* gs = static_cast<const T*>(a.b);
  T* guv = static_cast<T*>(a.out);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    const Pack<T> u = load16(uv + row * 2 * a.f + c);
    const Pack<T> v = load16(uv + row * 2 * a.f + a.f + c);
    const Pack<T> g = load16(gs + row * a.f + c);
    Pack<T> gu, gv;
#pragma unroll
    for (int i = 0; i < VN; ++i) {
      const float uf = to_f(u.v[i]), vf = to_f(v.v[i]), gf = to_f(g.v[i]);
      float guf, gvf;
      swiglu_bwd_f(uf, vf, gf, guf, gvf);
      gu.v[i] = from_f<T>(guf);
      gv.v[i] = from_f<T>(gvf);
    }
    store16(guv + row * 2 * a.f + c, gu);
    store16(guv + row * 2 * a.f + a.f + c, gv);
  }
}

// Squared ReLU (the block of the paper's experiments): s = relu(u)^2 and its
// backward gu = gs * 2 relu(u); u, s, gs, gu are [rows, f].
template <typename T>
__global__ __launch_bounds__(256) void ld_relu2_fwd_k(EltArgs a) {
  constexpr int VN = Pack<T>::N;
  const int64_t chunks = a.f / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const T* u = static_cast<const T*>(a.a);
  T* s = static_cast<T*>(a.out);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    const Pack<T> x = load16(u + row * a.f + c);
    Pack<T> o;
#pragma unroll
    for (int i = 0; i < VN; ++i) {
      const float r = fmaxf(to_f(x.v[i]), 0.f);
      o.v[i] = from_f<T>(r * r);
    }
    store16(s + row * a.f + c, o);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void ld_relu2_bwd_k(EltArgs a) {
  constexpr int VN = Pack<T>::N;
  const int64_t chunks = a.f / VN;
  const int64_t total = row_count(a.rc) * chunks;
  const T* u = static_cast<const T*>(a.a);
  const T* gs = static_cast<const T*>(a.b);
  T* gu = static_cast<T*>(a.out);
  for (int64_t id = blockIdx.x * 256ll + threadIdx.x; id < total; id += gridDim.x * 256ll) {
    const int64_t row = id / chunks, c = (id % chunks) * VN;
    const Pack<T> x = load16(u + row * a.f + c);
    const Pack<T> g = load16(gs + row * a.f + c);
    Pack<T> o;
#pragma unroll
    for (int i = 0; i < VN; ++i) o.v[i] = from_f<T>(to_f(g.v[i]) * 2.f * fmaxf(to_f(x.v[i]), 0.f));
    store16(gu + row * a.f + c, o);
  }
}

int elt_grid(int64_t total_chunks) {
  int64_t g = (total_chunks + 255) / 256;
  if (g > 8192) g = 8192;
  if (g < 1) g = 1;
  return static_cast<int>(g);
}

template <int VN>
int nch_bucket(int d) {
  const int nch = (d + 64 * VN - 1) / (64 * VN);
  return nch <= 1 ? 1 : nch <= 2 ? 2 : nch <= 4 ? 4 : 8;
}

template <typename TS, typename TY>
hipError_t rms_fwd_t(const RmsFwdArgs& a, hipStream_t s) {
  constexpr int VN = std::is_same<TY, bf16>::value ? 8 : 4;
  const int64_t max_rows = a.rc.rows;
  if (max_rows == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((max_rows + 3) / 4));
#define LD_RF(N) \
  case N: hipLaunchKernelGGL((ld_rmsnorm_fwd_k<TS, TY, VN, N>), grid, dim3(256), 0, s, a); break;
  switch (nch_bucket<VN>(a.d)) {
    LD_RF(1) LD_RF(2) LD_RF(4) LD_RF(8)
  }
#undef LD_RF
  return hipGetLastError();
}

template <typename TX, typename TY, typename TR, typename TO>
hipError_t rms_bwd_t(const RmsBwdArgs& a, float* dg, hipStream_t s) {
  constexpr int VN = std::is_same<TY, bf16>::value ? 8 : 4;
  const int64_t nblk = rmsnorm_bwd_blocks(a.rc.rows);
  // chunks of VN columns per thread of the 256
  const int nch = (a.d + 256 * VN - 1) / (256 * VN);
#define LD_RB(N) \
  case N: hipLaunchKernelGGL((ld_rmsnorm_bwd_k<TX, TY, TR, TO, VN, N>), dim3(nblk), dim3(256), 0, s, a); break;
  switch (nch <= 1 ? 1 : 2) {
    LD_RB(1) LD_RB(2)
  }
#undef LD_RB
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ld_dg_reduce_k, dim3((a.d + kDgCols - 1) / kDgCols), dim3(kDgCols * kDgGroups), 0, s, a.dg_part, nblk,
                     a.d, dg);
  return hipGetLastError();
}

// bf16 configuration: x, gres and gx each bf16 or float32
template <typename TX, typename TR>
hipError_t rms_bwd_bf16_o(const RmsBwdArgs& a, float* dg, hipStream_t s) {
  return a.gx_f32 ? rms_bwd_t<TX, bf16, TR, float>(a, dg, s) : rms_bwd_t<TX, bf16, TR, bf16>(a, dg, s);
}
template <typename TX>
hipError_t rms_bwd_bf16_r(const RmsBwdArgs& a, float* dg, hipStream_t s) {
  return a.gres_f32 ? rms_bwd_bf16_o<TX, float>(a, dg, s) : rms_bwd_bf16_o<TX, bf16>(a, dg, s);
}

}  // namespace

int64_t rmsnorm_bwd_blocks(int64_t max_rows) {
  const int64_t n = (max_rows + kBwdRowsPerBlock - 1) / kBwdRowsPerBlock;
  return n < 1 ? 1 : n;
}

hipError_t launch_masks(const MaskArgs& a, hipStream_t s) {
  int threads = ((a.batch + 63) / 64) * 64;
  if (threads > 1024) threads = 1024;
  hipLaunchKernelGGL(ld_mask_compact, dim3(a.n_layers * a.n_masks), dim3(threads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_zero_f32(const ZeroArgs& a, hipStream_t s) {
  int64_t most = 0;
  for (int i = 0; i < a.count; ++i) most = a.n[i] > most ? a.n[i] : most;
  if (most == 0) return hipSuccess;
  hipLaunchKernelGGL(ld_zero_f32_k, dim3(elt_grid(most / 4 + 1)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather(int dtype, const RowsArgs& a, hipStream_t s) {
  const int vn = dtype == LD_BF16 ? 8 : 4;
  const int grid = elt_grid(a.rc.rows * (a.d / vn));
  if (dtype == LD_BF16 && a.src_f32)
    hipLaunchKernelGGL((ld_gather_rows_k<float, bf16>), dim3(grid), dim3(256), 0, s, a);
  else if (dtype == LD_BF16)
    hipLaunchKernelGGL((ld_gather_rows_k<bf16, bf16>), dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((ld_gather_rows_k<float, float>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_convert(const void* src, void* dst, int64_t n, int to_f32, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 8) return hipErrorInvalidValue;
  const int grid = elt_grid(n / 8);
  if (to_f32)
    hipLaunchKernelGGL((ld_convert_k<bf16, float>), dim3(grid), dim3(256), 0, s, static_cast<const bf16*>(src),
                       static_cast<float*>(dst), n / 8);
  else
    hipLaunchKernelGGL((ld_convert_k<float, bf16>), dim3(grid), dim3(256), 0, s, static_cast<const float*>(src),
                       static_cast<bf16*>(dst), n / 8);
  return hipGetLastError();
}

hipError_t launch_scatter_add(int dtype, const RowsArgs& a, hipStream_t s) {
  const int vn = dtype == LD_BF16 ? 8 : 4;
  const int grid = elt_grid(a.rc.rows * (a.d / vn));
  if (dtype == LD_BF16)
    hipLaunchKernelGGL(ld_scatter_add_rows_k<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ld_scatter_add_rows_k<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_fwd(int dtype, const RmsFwdArgs& a, hipStream_t s) {
  if (dtype != LD_BF16) return rms_fwd_t<float, float>(a, s);
  return a.x_f32 ? rms_fwd_t<float, bf16>(a, s) : rms_fwd_t<bf16, bf16>(a, s);
}

hipError_t launch_rmsnorm_bwd(int dtype, const RmsBwdArgs& a, float* dg, hipStream_t s) {
  if (dtype != LD_BF16) return rms_bwd_t<float, float, float, float>(a, dg, s);
  return a.x_f32 ? rms_bwd_bf16_r<float>(a, dg, s) : rms_bwd_bf16_r<bf16>(a, dg, s);
}

hipError_t launch_relu2_fwd(int dtype, const EltArgs& a, hipStream_t s) {
  const int grid = elt_grid(a.rc.rows * (a.f / (dtype == LD_BF16 ? Pack<bf16>::N : Pack<float>::N)));
  if (a.rc.rows == 0) return hipSuccess;
  if (dtype == LD_BF16)
    hipLaunchKernelGGL(ld_relu2_fwd_k<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ld_relu2_fwd_k<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_relu2_bwd(int dtype, const EltArgs& a, hipStream_t s) {
  const int grid = elt_grid(a.rc.rows * (a.f / (dtype == LD_BF16 ? Pack<bf16>::N : Pack<float>::N)));
  if (a.rc.rows == 0) return hipSuccess;
  if (dtype == LD_BF16)
    hipLaunchKernelGGL(ld_relu2_bwd_k<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ld_relu2_bwd_k<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_swiglu_fwd(int dtype, const EltArgs& a, hipStream_t s) {
  const int vn = dtype == LD_BF16 ? 8 : 4;
  const int grid = elt_grid(a.rc.rows * (a.f / vn));
  if (dtype == LD_BF16)
    hipLaunchKernelGGL(ld_swiglu_fwd_k<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ld_swiglu_fwd_k<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(int dtype, const EltArgs& a, hipStream_t s) {
  const int vn = dtype == LD_BF16 ? 8 : 4;
  const int grid = elt_grid(a.rc.rows * (a.f / vn));
  if (dtype == LD_BF16)
    hipLaunchKernelGGL(ld_swiglu_bwd_k<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ld_swiglu_bwd_k<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ld

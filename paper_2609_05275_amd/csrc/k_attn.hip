// Causal multi-head attention, forward and backward, on kept sequences only.
//
// bf16 path (d_head 64 or 128), gfx950 MFMA v_mfma_f32_32x32x16_bf16:
//   Forward: one workgroup per (128-row query tile, head, kept sequence), four
//   waves of 32 query rows.  Scores are formed transposed, S^T = K Q^T, so a
//   lane owns one query row (its column of the 32x32 accumulator) and holds
//   16 of the block's keys; the softmax statistics are per lane, with one
//   exchange between the two half-waves for the running maximum.  The
//   accumulator layout (row 8*(v/4) + 4*(lane/32) + v%4) is reused directly as
//   the B operand of O^T += V^T P^T: the keys a lane holds are a permutation of
//   the MFMA k index, and V^T is read from LDS in the same permutation (two
//   8-byte reads per fragment).  K is staged [key][d], V transposed [d][key].
//   Online softmax in base 2, fp32; O normalised at the end and the natural
//   log-sum-exp saved per row.
//   Backward (no float atomics): delta = rowsum(dO * O); a dK/dV kernel per
//   (128-key tile, head, sequence) walks the query blocks at and after the
//   diagonal recomputing P from the saved log-sum-exp; a dQ kernel per
//   (128-row query tile, head, sequence) walks the key blocks up to the
//   diagonal.  Heavy (late) query tiles are scheduled first.
// fp32 path: plain SIMT kernels, one thread per query (or key) row, used by
// the fp32 configuration only.
#include "ld_internal.h"

namespace ld {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ int seq_count(const AttnArgs& a) {
  return a.dev_count ? *a.dev_count : a.n_seq;
}

__device__ __forceinline__ floatx16 mfma(const bf16x8& a, const bf16x8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 load8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = static_cast<bf16>(0.f);
  return z;
}

// Two 4-element pieces of an LDS row -> one 8-element fragment.
__device__ __forceinline__ bf16x8 load4x2(const bf16* lo, const bf16* hi) {
  const uint2 a = *reinterpret_cast<const uint2*>(lo);
  const uint2 b = *reinterpret_cast<const uint2*>(hi);
  uint4 u = make_uint4(a.x, a.y, b.x, b.y);
  return *reinterpret_cast<const bf16x8*>(&u);
}

__device__ __forceinline__ uint32_t half_of(const uint4& v, int i) {
  const uint32_t w = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
  return (i & 1) ? (w >> 16) : (w & 0xffffu);
}

// Stage rows [r0, r0+ROWS) x DH of a strided bf16 matrix into LDS, both as
// [row][d] (pitch DH+8) when `direct` is set and transposed as [d][row]
// (pitch ROWS+8) when `trans` is set.  Rows at or past `limit` are zero.
template <int ROWS, int DH>
__device__ __forceinline__ void stage_rows(const bf16* src, int64_t ld, int r0, int limit,
                                           bf16* direct, bf16* trans, int tid) {
  if (direct) {
    for (int c = tid; c < ROWS * DH / 8; c += 256) {
      const int r = c / (DH / 8), dc = (c % (DH / 8)) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (r0 + r < limit) v = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(r0 + r) * ld + dc);
      *reinterpret_cast<uint4*>(direct + r * (DH + 8) + dc) = v;
    }
  }
  if (trans) {
    for (int c = tid; c < (ROWS / 4) * (DH / 8); c += 256) {
      const int rg = (c / (DH / 8)) * 4, dc = (c % (DH / 8)) * 8;
      uint4 v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        v[k] = make_uint4(0, 0, 0, 0);
        if (r0 + rg + k < limit)
          v[k] = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(r0 + rg + k) * ld + dc);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        uint2 o;
        o.x = half_of(v[0], i) | (half_of(v[1], i) << 16);
        o.y = half_of(v[2], i) | (half_of(v[3], i) << 16);
        *reinterpret_cast<uint2*>(trans + (dc + i) * (ROWS + 8) + rg) = o;
      }
    }
  }
}

// ---------------------------------------------------------------- forward

constexpr int FQ = 128, FKV = 64;

template <int DH>
__global__ __launch_bounds__(256) void ld_attn_fwd_bf16(AttnArgs a) {
  __shared__ __align__(16) bf16 Ks[FKV * (DH + 8)];
  __shared__ __align__(16) bf16 Vt[DH * (FKV + 8)];
  const int S = a.S, H = a.H;
  const int n_qt = (S + FQ - 1) / FQ;
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.x);
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hf = lane >> 5, cl = lane & 31;
  const int q0 = qt * FQ, qw = q0 + wave * 32, qrow = qw + cl;
  const bool active = qw < S;
  const int64_t ldq = 3ll * H * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  const bf16* Kp = base + static_cast<int64_t>(H) * DH + head * DH;
  const bf16* Vp = base + 2ll * H * DH + head * DH;
  const float sl2 = a.scale * kLog2e;

  bf16x8 qf[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks)
    qf[ks] = qrow < S ? load8(Qp + static_cast<int64_t>(qrow) * ldq + ks * 16 + hf * 8) : zero8();
  floatx16 o[DH / 32];
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m = -INFINITY, l = 0.f;

  const int kv_end = min(S, q0 + FQ);
  for (int k0 = 0; k0 < kv_end; k0 += FKV) {
    stage_rows<FKV, DH>(Kp, ldq, k0, S, Ks, nullptr, tid);
    stage_rows<FKV, DH>(Vp, ldq, k0, S, nullptr, Vt, tid);
    __syncthreads();
    if (active && k0 <= qw + 31) {
      floatx16 s[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int v = 0; v < 16; ++v) s[kh][v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < DH / 16; ++ks)
          s[kh] = mfma(load8(Ks + (kh * 32 + cl) * (DH + 8) + ks * 16 + hf * 8), qf[ks], s[kh]);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = k0 + kh * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
          float x = s[kh][v] * sl2;
          if (key > qrow || key >= S) x = -INFINITY;
          s[kh][v] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m, mx);
      const float alpha = exp2f(m - m_new);
      m = m_new;
      float ls = 0.f;
      bf16x8 pb[2][2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float p = exp2f(s[kh][v] - m_new);
          ls += p;
          pb[kh][v >> 3][v & 7] = static_cast<bf16>(p);
        }
      l = l * alpha + ls;
#pragma unroll
      for (int db = 0; db < DH / 32; ++db) {
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
        const bf16* vrow = Vt + (db * 32 + cl) * (FKV + 8);
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int kb = kh * 32 + 16 * c + 4 * hf;
            o[db] = mfma(load4x2(vrow + kb, vrow + kb + 8), pb[kh][c], o[db]);
          }
      }
    }
    __syncthreads();
  }
  const float lt = l + __shfl_xor(l, 32, 64);
  if (active && qrow < S) {
    const float inv = 1.f / lt;
    bf16* Op = static_cast<bf16*>(a.out) + (static_cast<int64_t>(seq) * S + qrow) * (static_cast<int64_t>(H) * DH) + head * DH;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        __attribute__((aligned(8))) bf16 t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) t[i] = static_cast<bf16>(o[db][4 * g + i] * inv);
        *reinterpret_cast<uint2*>(Op + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(t);
      }
    if (hf == 0) a.lse[(static_cast<int64_t>(seq) * H + head) * S + qrow] = (m + log2f(lt)) * kLn2;
  }
}

// --------------------------------------------------------------- backward

template <typename T, int DH>
__global__ __launch_bounds__(256) void ld_attn_delta(AttnArgs a) {
  const int64_t rows = static_cast<int64_t>(seq_count(a)) * a.S * a.H;
  const int64_t id = blockIdx.x * 256ll + threadIdx.x;
  if (id >= rows) return;
  const int64_t tok = id / a.H;
  const int head = static_cast<int>(id % a.H);
  const int64_t ld = static_cast<int64_t>(a.H) * DH;
  const T* o = static_cast<const T*>(a.o) + tok * ld + head * DH;
  const T* go = static_cast<const T*>(a.go) + tok * ld + head * DH;
  float s = 0.f;
  for (int i = 0; i < DH; ++i) s = __builtin_fmaf(static_cast<float>(o[i]), static_cast<float>(go[i]), s);
  const int64_t seq = tok / a.S, q = tok % a.S;
  a.delta[(seq * a.H + head) * a.S + q] = s;
}

constexpr int BQ = 32;       // query rows per step of the dK/dV kernel
constexpr int BKEYS = 128;   // keys per dK/dV workgroup (4 waves x 32)

template <int DH>
__global__ __launch_bounds__(256) void ld_attn_bwd_dkdv_bf16(AttnArgs a) {
  __shared__ __align__(16) bf16 Qs[BQ * (DH + 8)];
  __shared__ __align__(16) bf16 Qt[DH * (BQ + 8)];
  __shared__ __align__(16) bf16 Os[BQ * (DH + 8)];   // dO [q][d]
  __shared__ __align__(16) bf16 Ot[DH * (BQ + 8)];   // dO^T [d][q]
  __shared__ float lse_s[BQ], del_s[BQ];
  const int S = a.S, H = a.H;
  const int n_kt = (S + BKEYS - 1) / BKEYS;
  const int kt = static_cast<int>(blockIdx.x);  // early key tiles see the most queries
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  (void)n_kt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hf = lane >> 5, cl = lane & 31;
  const int k0 = kt * BKEYS, kw = k0 + wave * 32, key = kw + cl;
  const bool active = kw < S;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  const bf16* Kp = base + static_cast<int64_t>(H) * DH + head * DH;
  const bf16* Vp = base + 2ll * H * DH + head * DH;
  const bf16* dOp = static_cast<const bf16*>(a.go) + static_cast<int64_t>(seq) * S * ldo + head * DH;
  const float* lse = a.lse + (static_cast<int64_t>(seq) * H + head) * S;
  const float* del = a.delta + (static_cast<int64_t>(seq) * H + head) * S;
  const float sl2 = a.scale * kLog2e;

  bf16x8 kf[DH / 16], vf[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) {
    kf[ks] = key < S ? load8(Kp + static_cast<int64_t>(key) * ldq + ks * 16 + hf * 8) : zero8();
    vf[ks] = key < S ? load8(Vp + static_cast<int64_t>(key) * ldq + ks * 16 + hf * 8) : zero8();
  }
  floatx16 dv[DH / 32], dk[DH / 32];
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) dv[db][v] = dk[db][v] = 0.f;

  for (int q0 = k0; q0 < S; q0 += BQ) {
    stage_rows<BQ, DH>(Qp, ldq, q0, S, Qs, Qt, tid);
    stage_rows<BQ, DH>(dOp, ldo, q0, S, Os, Ot, tid);
    if (tid < BQ) {
      const bool ok = q0 + tid < S;
      lse_s[tid] = ok ? lse[q0 + tid] * kLog2e : 0.f;
      del_s[tid] = ok ? del[q0 + tid] : 0.f;
    }
    __syncthreads();
    if (active && kw <= q0 + BQ - 1) {
      floatx16 s, dp;
#pragma unroll
      for (int v = 0; v < 16; ++v) s[v] = dp[v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        s = mfma(load8(Qs + cl * (DH + 8) + ks * 16 + hf * 8), kf[ks], s);
        dp = mfma(load8(Os + cl * (DH + 8) + ks * 16 + hf * 8), vf[ks], dp);
      }
      bf16x8 pb[2], db8[2];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int ql = 8 * (v >> 2) + 4 * hf + (v & 3);
        const int q = q0 + ql;
        float p = 0.f;
        if (q < S && key <= q) p = exp2f(s[v] * sl2 - lse_s[ql]);
        const float ds = p * (dp[v] - del_s[ql]);
        pb[v >> 3][v & 7] = static_cast<bf16>(p);
        db8[v >> 3][v & 7] = static_cast<bf16>(ds);
      }
#pragma unroll
      for (int db = 0; db < DH / 32; ++db) {
        const bf16* orow = Ot + (db * 32 + cl) * (BQ + 8);
        const bf16* qrow = Qt + (db * 32 + cl) * (BQ + 8);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int qb = 16 * c + 4 * hf;
          dv[db] = mfma(load4x2(orow + qb, orow + qb + 8), pb[c], dv[db]);
          dk[db] = mfma(load4x2(qrow + qb, qrow + qb + 8), db8[c], dk[db]);
        }
      }
    }
    __syncthreads();
  }
  if (active && key < S) {
    bf16* G = static_cast<bf16*>(a.out) + (static_cast<int64_t>(seq) * S + key) * ldq + head * DH;
    bf16* Gk = G + static_cast<int64_t>(H) * DH;
    bf16* Gv = G + 2ll * H * DH;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        __attribute__((aligned(8))) bf16 tk[4], tv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          tk[i] = static_cast<bf16>(dk[db][4 * g + i] * a.scale);
          tv[i] = static_cast<bf16>(dv[db][4 * g + i]);
        }
        *reinterpret_cast<uint2*>(Gk + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(tk);
        *reinterpret_cast<uint2*>(Gv + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(tv);
      }
  }
}

template <int DH>
__global__ __launch_bounds__(256) void ld_attn_bwd_dq_bf16(AttnArgs a) {
  __shared__ __align__(16) bf16 Ks[FKV * (DH + 8)];
  __shared__ __align__(16) bf16 Kt[DH * (FKV + 8)];
  __shared__ __align__(16) bf16 Vs[FKV * (DH + 8)];
  const int S = a.S, H = a.H;
  const int n_qt = (S + FQ - 1) / FQ;
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.x);
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hf = lane >> 5, cl = lane & 31;
  const int q0 = qt * FQ, qw = q0 + wave * 32, qrow = qw + cl;
  const bool active = qw < S;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  const bf16* Kp = base + static_cast<int64_t>(H) * DH + head * DH;
  const bf16* Vp = base + 2ll * H * DH + head * DH;
  const bf16* dOp = static_cast<const bf16*>(a.go) + static_cast<int64_t>(seq) * S * ldo + head * DH;
  const float sl2 = a.scale * kLog2e;
  const bool qok = qrow < S;
  const int64_t srow = (static_cast<int64_t>(seq) * H + head) * S + (qok ? qrow : 0);
  const float lse2 = qok ? a.lse[srow] * kLog2e : 0.f;
  const float dl = qok ? a.delta[srow] : 0.f;

  bf16x8 qf[DH / 16], of[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) {
    qf[ks] = qok ? load8(Qp + static_cast<int64_t>(qrow) * ldq + ks * 16 + hf * 8) : zero8();
    of[ks] = qok ? load8(dOp + static_cast<int64_t>(qrow) * ldo + ks * 16 + hf * 8) : zero8();
  }
  floatx16 dq[DH / 32];
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) dq[db][v] = 0.f;

  const int kv_end = min(S, q0 + FQ);
  for (int k0 = 0; k0 < kv_end; k0 += FKV) {
    stage_rows<FKV, DH>(Kp, ldq, k0, S, Ks, Kt, tid);
    stage_rows<FKV, DH>(Vp, ldq, k0, S, Vs, nullptr, tid);
    __syncthreads();
    if (active && k0 <= qw + 31) {
      bf16x8 dsb[2][2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        floatx16 s, dp;
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = dp[v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < DH / 16; ++ks) {
          s = mfma(load8(Ks + (kh * 32 + cl) * (DH + 8) + ks * 16 + hf * 8), qf[ks], s);
          dp = mfma(load8(Vs + (kh * 32 + cl) * (DH + 8) + ks * 16 + hf * 8), of[ks], dp);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = k0 + kh * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
          float p = 0.f;
          if (qok && key <= qrow) p = exp2f(s[v] * sl2 - lse2);
          dsb[kh][v >> 3][v & 7] = static_cast<bf16>(p * (dp[v] - dl));
        }
      }
#pragma unroll
      for (int db = 0; db < DH / 32; ++db) {
        const bf16* krow = Kt + (db * 32 + cl) * (FKV + 8);
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int kb = kh * 32 + 16 * c + 4 * hf;
            dq[db] = mfma(load4x2(krow + kb, krow + kb + 8), dsb[kh][c], dq[db]);
          }
      }
    }
    __syncthreads();
  }
  if (active && qok) {
    bf16* G = static_cast<bf16*>(a.out) + (static_cast<int64_t>(seq) * S + qrow) * ldq + head * DH;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        __attribute__((aligned(8))) bf16 t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) t[i] = static_cast<bf16>(dq[db][4 * g + i] * a.scale);
        *reinterpret_cast<uint2*>(G + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(t);
      }
  }
}

// ------------------------------------------------------------ fp32 (SIMT)

constexpr int ST = 64;  // rows per workgroup and keys per LDS tile

template <int DH>
__global__ __launch_bounds__(64) void ld_attn_fwd_f32(AttnArgs a) {
  __shared__ float Ks[ST][DH], Vs[ST][DH];
  const int S = a.S, H = a.H;
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  const int q0 = blockIdx.x * ST, q = q0 + threadIdx.x;
  const int64_t ldq = 3ll * H * DH;
  const float* base = static_cast<const float*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  float qv[DH], o[DH];
  for (int i = 0; i < DH; ++i) {
    qv[i] = q < S ? base[static_cast<int64_t>(q) * ldq + head * DH + i] : 0.f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int kv_end = min(S, q0 + ST);
  for (int k0 = 0; k0 < kv_end; k0 += ST) {
    for (int e = threadIdx.x; e < ST * DH; e += ST) {
      const int r = e / DH, c = e % DH;
      const bool ok = k0 + r < S;
      Ks[r][c] = ok ? base[static_cast<int64_t>(k0 + r) * ldq + H * DH + head * DH + c] : 0.f;
      Vs[r][c] = ok ? base[static_cast<int64_t>(k0 + r) * ldq + 2 * H * DH + head * DH + c] : 0.f;
    }
    __syncthreads();
    for (int j = 0; j < ST; ++j) {
      const int key = k0 + j;
      if (key > q || key >= S) break;
      float s = 0.f;
      for (int i = 0; i < DH; ++i) s = __builtin_fmaf(qv[i], Ks[j][i], s);
      s *= a.scale;
      const float m_new = fmaxf(m, s);
      const float alpha = expf(m - m_new), p = expf(s - m_new);
      l = l * alpha + p;
      for (int i = 0; i < DH; ++i) o[i] = o[i] * alpha + p * Vs[j][i];
      m = m_new;
    }
    __syncthreads();
  }
  if (q < S) {
    float* Op = static_cast<float*>(a.out) + (static_cast<int64_t>(seq) * S + q) * (static_cast<int64_t>(H) * DH) + head * DH;
    for (int i = 0; i < DH; ++i) Op[i] = o[i] / l;
    a.lse[(static_cast<int64_t>(seq) * H + head) * S + q] = m + logf(l);
  }
}

template <int DH>
__global__ __launch_bounds__(64) void ld_attn_bwd_dq_f32(AttnArgs a) {
  __shared__ float Ks[ST][DH], Vs[ST][DH];
  const int S = a.S, H = a.H;
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  const int q0 = blockIdx.x * ST, q = q0 + threadIdx.x;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const float* base = static_cast<const float*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const float* go = static_cast<const float*>(a.go) + static_cast<int64_t>(seq) * S * ldo;
  float qv[DH], dov[DH], dq[DH];
  for (int i = 0; i < DH; ++i) {
    qv[i] = q < S ? base[static_cast<int64_t>(q) * ldq + head * DH + i] : 0.f;
    dov[i] = q < S ? go[static_cast<int64_t>(q) * ldo + head * DH + i] : 0.f;
    dq[i] = 0.f;
  }
  const int64_t srow = (static_cast<int64_t>(seq) * H + head) * S + (q < S ? q : 0);
  const float lse = a.lse[srow], dl = a.delta[srow];
  const int kv_end = min(S, q0 + ST);
  for (int k0 = 0; k0 < kv_end; k0 += ST) {
    for (int e = threadIdx.x; e < ST * DH; e += ST) {
      const int r = e / DH, c = e % DH;
      const bool ok = k0 + r < S;
      Ks[r][c] = ok ? base[static_cast<int64_t>(k0 + r) * ldq + H * DH + head * DH + c] : 0.f;
      Vs[r][c] = ok ? base[static_cast<int64_t>(k0 + r) * ldq + 2 * H * DH + head * DH + c] : 0.f;
    }
    __syncthreads();
    for (int j = 0; j < ST; ++j) {
      const int key = k0 + j;
      if (key > q || key >= S) break;
      float s = 0.f, dp = 0.f;
      for (int i = 0; i < DH; ++i) {
        s = __builtin_fmaf(qv[i], Ks[j][i], s);
        dp = __builtin_fmaf(dov[i], Vs[j][i], dp);
      }
      const float p = expf(s * a.scale - lse);
      const float ds = p * (dp - dl);
      for (int i = 0; i < DH; ++i) dq[i] = __builtin_fmaf(ds, Ks[j][i], dq[i]);
    }
    __syncthreads();
  }
  if (q < S) {
    float* G = static_cast<float*>(a.out) + (static_cast<int64_t>(seq) * S + q) * ldq + head * DH;
    for (int i = 0; i < DH; ++i) G[i] = dq[i] * a.scale;
  }
}

template <int DH>
__global__ __launch_bounds__(64) void ld_attn_bwd_dkdv_f32(AttnArgs a) {
  __shared__ float Qs[ST][DH], Os[ST][DH], ls[ST], dls[ST];
  const int S = a.S, H = a.H;
  const int head = blockIdx.y, seq = blockIdx.z;
  if (seq >= seq_count(a)) return;
  const int k0 = blockIdx.x * ST, key = k0 + threadIdx.x;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const float* base = static_cast<const float*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const float* go = static_cast<const float*>(a.go) + static_cast<int64_t>(seq) * S * ldo;
  const float* lse = a.lse + (static_cast<int64_t>(seq) * H + head) * S;
  const float* del = a.delta + (static_cast<int64_t>(seq) * H + head) * S;
  float kv[DH], vv[DH], dk[DH], dv[DH];
  for (int i = 0; i < DH; ++i) {
    kv[i] = key < S ? base[static_cast<int64_t>(key) * ldq + H * DH + head * DH + i] : 0.f;
    vv[i] = key < S ? base[static_cast<int64_t>(key) * ldq + 2 * H * DH + head * DH + i] : 0.f;
    dk[i] = dv[i] = 0.f;
  }
  for (int qb = k0; qb < S; qb += ST) {
    for (int e = threadIdx.x; e < ST * DH; e += ST) {
      const int r = e / DH, c = e % DH;
      const bool ok = qb + r < S;
      Qs[r][c] = ok ? base[static_cast<int64_t>(qb + r) * ldq + head * DH + c] : 0.f;
      Os[r][c] = ok ? go[static_cast<int64_t>(qb + r) * ldo + head * DH + c] : 0.f;
    }
    if (threadIdx.x < ST) {
      const bool ok = qb + threadIdx.x < S;
      ls[threadIdx.x] = ok ? lse[qb + threadIdx.x] : 0.f;
      dls[threadIdx.x] = ok ? del[qb + threadIdx.x] : 0.f;
    }
    __syncthreads();
    if (key < S) {
      for (int j = 0; j < ST; ++j) {
        const int q = qb + j;
        if (q >= S) break;
        if (q < key) continue;
        float s = 0.f, dp = 0.f;
        for (int i = 0; i < DH; ++i) {
          s = __builtin_fmaf(Qs[j][i], kv[i], s);
          dp = __builtin_fmaf(Os[j][i], vv[i], dp);
        }
        const float p = expf(s * a.scale - ls[j]);
        const float ds = p * (dp - dls[j]);
        for (int i = 0; i < DH; ++i) {
          dv[i] = __builtin_fmaf(p, Os[j][i], dv[i]);
          dk[i] = __builtin_fmaf(ds, Qs[j][i], dk[i]);
        }
      }
    }
    __syncthreads();
  }
  if (key < S) {
    float* G = static_cast<float*>(a.out) + (static_cast<int64_t>(seq) * S + key) * ldq + head * DH;
    for (int i = 0; i < DH; ++i) {
      G[H * DH + i] = dk[i] * a.scale;
      G[2 * H * DH + i] = dv[i];
    }
  }
}

template <int DH>
hipError_t fwd_dh(int dtype, const AttnArgs& a, hipStream_t s) {
  if constexpr (DH >= 64) {
    if (dtype == LD_BF16) {
      const dim3 grid((a.S + FQ - 1) / FQ, a.H, a.n_seq);
      hipLaunchKernelGGL(ld_attn_fwd_bf16<DH>, grid, dim3(256), 0, s, a);
      return hipGetLastError();
    }
  }
  if constexpr (DH <= 64) {
    const dim3 grid((a.S + ST - 1) / ST, a.H, a.n_seq);
    hipLaunchKernelGGL(ld_attn_fwd_f32<DH>, grid, dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

template <int DH>
hipError_t bwd_dh(int dtype, const AttnArgs& a, hipStream_t s) {
  const int64_t rows = static_cast<int64_t>(a.n_seq) * a.S * a.H;
  const dim3 dgrid(static_cast<unsigned>((rows + 255) / 256));
  if constexpr (DH >= 64) {
    if (dtype == LD_BF16) {
      hipLaunchKernelGGL((ld_attn_delta<bf16, DH>), dgrid, dim3(256), 0, s, a);
      hipLaunchKernelGGL(ld_attn_bwd_dkdv_bf16<DH>, dim3((a.S + BKEYS - 1) / BKEYS, a.H, a.n_seq),
                         dim3(256), 0, s, a);
      hipLaunchKernelGGL(ld_attn_bwd_dq_bf16<DH>, dim3((a.S + FQ - 1) / FQ, a.H, a.n_seq),
                         dim3(256), 0, s, a);
      return hipGetLastError();
    }
  }
  if constexpr (DH <= 64) {
    hipLaunchKernelGGL((ld_attn_delta<float, DH>), dgrid, dim3(256), 0, s, a);
    const dim3 grid((a.S + ST - 1) / ST, a.H, a.n_seq);
    hipLaunchKernelGGL(ld_attn_bwd_dkdv_f32<DH>, grid, dim3(64), 0, s, a);
    hipLaunchKernelGGL(ld_attn_bwd_dq_f32<DH>, grid, dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

const char* attn_fwd_kernel_name(int dtype) {
  return dtype == LD_BF16 ? "ld_attn_fwd_bf16" : "ld_attn_fwd_f32";
}

hipError_t launch_attn_fwd(int dtype, const AttnArgs& a, hipStream_t s) {
  if (a.n_seq <= 0) return hipSuccess;
  if (dtype == LD_BF16) {
    if (a.dh == 64) return fwd_dh<64>(dtype, a, s);
    if (a.dh == 128) return fwd_dh<128>(dtype, a, s);
    return hipErrorInvalidValue;
  }
  switch (a.dh) {
    case 16: return fwd_dh<16>(dtype, a, s);
    case 32: return fwd_dh<32>(dtype, a, s);
    case 64: return fwd_dh<64>(dtype, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attn_bwd(int dtype, const AttnArgs& a, hipStream_t s) {
  if (a.n_seq <= 0) return hipSuccess;
  if (dtype == LD_BF16) {
    if (a.dh == 64) return bwd_dh<64>(dtype, a, s);
    if (a.dh == 128) return bwd_dh<128>(dtype, a, s);
    return hipErrorInvalidValue;
  }
  switch (a.dh) {
    case 16: return bwd_dh<16>(dtype, a, s);
    case 32: return bwd_dh<32>(dtype, a, s);
    case 64: return bwd_dh<64>(dtype, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ld

// Causal multi-head attention, forward and backward, on kept sequences only.
//
// bf16 path (d_head 64 or 128), gfx950 MFMA v_mfma_f32_32x32x16_bf16.  Every
// kernel streams 64-row blocks of [row][d] bf16 (keys and values, or queries
// and output gradients) from global memory straight into a four-stage LDS
// ring with buffer loads that have an LDS destination; the 16-byte chunks of
// a row are XOR-swizzled by the row so that plain fragment reads and the
// transposing reads (ds_read_b64_tr_b16) are bank-conflict free.  Scores are
// formed with the streamed rows as the MFMA A operand, so a lane owns one
// column (the wave's fixed query or key) and 16 streamed rows; that
// accumulator layout (row 8*(v/4) + 4*(lane/32) + v%4) is reused directly as
// the B operand of the next product, whose A operand (V^T, K^T, dO^T, Q^T) is
// read transposed from the same [row][d] block in the same row permutation.
//   Forward: one workgroup per (256-row query tile, head, kept sequence),
//   eight waves of 32 query rows; online softmax in base 2 with lazy
//   rescaling, O normalised at the end and the natural log-sum-exp saved.
//   Backward (no float atomics): a dQ kernel per (256-row query tile, head,
//   sequence) forms delta = rowsum(dO * O) of its rows first (stored negated
//   for the next kernel) and walks the key blocks up to the diagonal; then a
//   dK/dV kernel per (128-key tile, head, sequence) walks the query blocks at
//   and after the diagonal recomputing P from the saved log-sum-exp.  Heavy
//   causal tiles are scheduled first.
// fp32 path: plain SIMT kernels, one thread per query (or key) row, used by
// the fp32 configuration only.
#include <mutex>
#include <type_traits>

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

// The value of the lane 32 apart, as two halves of a wave: gfx950's
// v_permlane32_swap with x as both operands leaves the lower half's x in
// every lane of one result and the upper half's in the other, without an
// LDS round trip.
__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = static_cast<bf16>(0.f);
  return z;
}

// ---------------------------------------------------------------- forward

constexpr int FKV = 64;   // keys per streamed block
constexpr int FWQ = 256;            // forward: query rows per workgroup
constexpr int kFwdRowsPerWave = 32;  // forward: query rows per wave (8 waves)

// --------------------------------------------------------------- backward

// delta[seq, head, q] = -sum_d dO * O (float32, stored negated so that it can
// start the dP accumulation: dP - rowsum(dO * O) comes out of the MFMAs).
// One wave per token row of
// H*DH values: each pass reads 16 contiguous bytes per lane of O and dO (the
// row in 64*16-byte pieces), the DH/VN lanes of a head sum their products
// with butterfly shuffles, and the first lane of each head writes it.
template <typename T, int DH>
__global__ __launch_bounds__(256) void ld_attn_delta(AttnArgs a) {
  constexpr int VN = 16 / sizeof(T), G = DH / VN;  // elements per lane per pass, lanes per head
  static_assert(G >= 1 && 64 % G == 0, "a head spans whole lanes of a pass");
  const int64_t tokens = static_cast<int64_t>(seq_count(a)) * a.S;
  const int64_t tok = blockIdx.x * 4ll + (threadIdx.x >> 6);
  if (tok >= tokens) return;
  const int lane = threadIdx.x & 63;
  const int W = a.H * DH;
  const int64_t seq = tok / a.S, q = tok % a.S;
  const T* o = static_cast<const T*>(a.o) + tok * W;
  const T* go = static_cast<const T*>(a.go) + tok * W;
  for (int e0 = 0; e0 < W; e0 += 64 * VN) {
    const int e = e0 + lane * VN;
    float s = 0.f;
    if (e < W) {
      const uint4 ov = *reinterpret_cast<const uint4*>(o + e);
      const uint4 gv = *reinterpret_cast<const uint4*>(go + e);
      const T* op = reinterpret_cast<const T*>(&ov);
      const T* gp = reinterpret_cast<const T*>(&gv);
#pragma unroll
      for (int i = 0; i < VN; ++i) s = __builtin_fmaf(static_cast<float>(op[i]), static_cast<float>(gp[i]), s);
    }
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (e < W && lane % G == 0) a.delta[(seq * a.H + e / DH) * a.S + q] = -s;
  }
}

constexpr int BQ = 64;       // query rows per step of the dK/dV kernel
constexpr int DK_NST = 3;    // dK/dV ring stages (query blocks in LDS)

// Key groups of 32 per dK/dV workgroup: four, each served by a pair of waves.
constexpr int DK_GROUPS = 4;

// Q and dO blocks in the dK/dV ring are [64 q][DH] without padding, the
// 16-byte chunks of a row XOR-swizzled by row bits 0-3: 16 lanes reading one
// chunk of 16 consecutive rows, and the transposing reads (4 consecutive rows
// x 64 bytes per half-wave), both hit every bank once.
template <int DH>
__device__ __forceinline__ int qd_swz(int r) {
  if constexpr (DH == 128)
    return ((r & 3) << 2) | ((r >> 2) & 3);
  else
    return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}
template <int DH>
__device__ __forceinline__ int qd_off(int r, int d) {
  return r * DH + (((d >> 3) ^ qd_swz<DH>(r)) << 3) + (d & 7);
}

// One ring stage: the Q block, the dO block, then log-sum-exp and delta.
template <int DH>
constexpr int dk_stage_bytes() { return 4 * BQ * DH + 8 * BQ; }
// Loads per loading wave per stage: Q and dO in 1 KB pieces split over NW
// waves, plus the log-sum-exp and delta rows (every loading wave loads both:
// same bytes).
template <int DH, int NW>
constexpr int dk_loads() { return 2 * (BQ * DH * 2 / 1024) / NW + 2; }
// P exchange area after the ring: two slots (by half parity) x the key
// groups x 4 KB (64 lanes x 16 floats).
constexpr int kDkPSlot = DK_GROUPS * 4096;
constexpr int kDkPBytes = 2 * kDkPSlot;

typedef short v4s __attribute__((ext_vector_type(4)));

// LDS reads at a byte address (an LDS pointer as a 32-bit integer); constant
// parts of the address become instruction immediates.
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8_t;
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) const floatx4 lds_float4_t;
typedef __attribute__((address_space(3))) floatx4 lds_float4_w_t;
typedef __attribute__((address_space(3))) v4s lds_v4s_t;
__device__ __forceinline__ bf16x8 lds_frag(uint32_t addr) {
  return *reinterpret_cast<lds_bf16x8_t*>(static_cast<uintptr_t>(addr));
}
__device__ __forceinline__ void lds_put(uint32_t addr, const floatx4& v) {
  *reinterpret_cast<lds_float4_w_t*>(static_cast<uintptr_t>(addr)) = v;
}
__device__ __forceinline__ floatx4 lds_f4(uint32_t addr) {
  return *reinterpret_cast<lds_float4_t*>(static_cast<uintptr_t>(addr));
}
__device__ __forceinline__ v4s lds_tr(uint32_t addr) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_v4s_t*>(static_cast<uintptr_t>(addr)));
}
__device__ __forceinline__ bf16x8 tr_pair(const v4s& lo, const v4s& hi) {
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Waits for this wave's LDS accesses, then meets the workgroup.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// dK, dV.  A workgroup owns 128 keys in four groups of 32 and walks the
// 64-row query blocks from the diagonal to the end, in 32-query halves.  Each
// key group has two waves with different work, meant to share a SIMD (waves
// g and g + 4): wave A holds K and forms the scores S = Q K^T, P =
// 2^(s*scale*log2e - lse*log2e) (bf16) and dV^T += dO^T P; wave B holds V and
// forms dP - delta = dO V^T - delta, dS = P (dP - delta) and dK^T += Q^T dS.
// P (float32) goes from A to B through LDS, one half behind: in half u, A
// computes S(u) and P(u) and the dV product of half u-1, B computes dS(u-1),
// its dK product and dP(u).  A workgroup barrier ends every half; P has two
// slots per key group, by half parity, so A writes P(u) while B reads
// P(u-1).  Each wave spreads its vector work over its own MFMAs (A: the
// exponentials between its dV products, B: dS between its dP products),
// and with at most 256 registers each the two waves of a group share a
// SIMD, one's MFMAs filling the other's waits.  dV^T and dK^T take P and dS
// straight from the score layout (their rows are a fixed permutation of the
// MFMA k index), dO^T and Q^T come from the same [q][d] blocks through
// transposing reads (ds_read_b64_tr_b16) in that permutation.
//
// Q, dO, log-sum-exp and delta of each block go from global memory straight
// into a three-stage LDS ring (buffer loads with an LDS destination, issued
// by the B waves, see ld_internal.h): block j+2 is requested once block j-1
// is done, half a block into block j.  Fragment addresses are per-lane
// offsets moved by one stage per block; the loop has no branch around its
// MFMAs (query rows before a wave's keys are computed and masked to P = 0,
// blocks past the end read zeros, and waves past the end compute on zero
// K/V and store nothing).
template <int DH, int NG, bool AL>
__global__ __launch_bounds__(128 * NG) void ld_attn_bwd_dkdv_bf16(AttnArgs a) {
  constexpr int BKEYS = 32 * NG, SB = dk_stage_bytes<DH>(), NL = dk_loads<DH, NG>();
  constexpr int RPI = 512 / DH, LPR = 64 / RPI;   // rows per 1 KB load, lanes per row
  constexpr int NPW = (BQ * DH * 2 / 1024) / NG;  // 1 KB loads per loading wave per tensor
  constexpr int N = DH / 16, NDB = DH / 32;       // k steps of the score products, d blocks
  static_assert(DK_NST == 3, "stage arithmetic assumes a ring of three");
  static_assert(NG == DK_GROUPS, "the P area is sized for DK_GROUPS key groups");
  extern __shared__ __align__(16) char ring[];
  const int S = a.S, H = a.H;
  // grid (head, sequence, tile), tile slowest: early key tiles see the most
  // queries and go first
  const int kt = static_cast<int>(blockIdx.z);
  const int head = blockIdx.x, seq = blockIdx.y;
  if (seq >= seq_count(a)) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool role_b = wave >= NG;  // wave-uniform
  const int grp = wave & (NG - 1);
  const int hf = lane >> 5, cl = lane & 31;
  const int k0 = kt * BKEYS, kw = k0 + grp * 32, key = kw + cl;
  if (k0 >= S) return;  // the whole workgroup is past the end
  const bool active = kw < S;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  // wave A holds K, wave B holds V: the same fragment slots
  const bf16* KVp = base + (role_b ? 2ll : 1ll) * H * DH + head * DH;
  const bf16* dOp = static_cast<const bf16*>(a.go) + static_cast<int64_t>(seq) * S * ldo + head * DH;
  const float* lse = a.lse + (static_cast<int64_t>(seq) * H + head) * S;
  const float* del = a.delta + (static_cast<int64_t>(seq) * H + head) * S;
  const float sl2 = a.scale * kLog2e;
  const float al2 = AL ? alibi_slope(head, H) * kLog2e : 0.f;

  // K or V fragments of the wave's keys, loaded after the first ring block
  // was requested (one wait covers both).  They must have arrived before the
  // next ring loads are issued: the compiler does not see those loads, so a
  // wait of its own for these inside the loop would wait for all of them.
  bf16x8 kv[N];
  auto load_kv = [&]() {
#pragma unroll
    for (int ks = 0; ks < N; ++ks)
      kv[ks] = key < S ? load8(KVp + static_cast<int64_t>(key) * ldq + ks * 16 + hf * 8) : zero8();
#pragma unroll
    for (int ks = 0; ks < N; ++ks) asm volatile("" ::"v"(kv[ks]));
  };
  floatx16 acc[NDB];  // dV^T (wave A) or dK^T (wave B)
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[db][v] = 0.f;

  // Loads of query block qb into stage st, by the B waves.  Blocks past the
  // end (qb >= S) read zeros.
  const dma_rsrc rq = dma_make_rsrc(Qp, static_cast<int64_t>(S) * ldq * 2);
  const dma_rsrc ro = dma_make_rsrc(dOp, static_cast<int64_t>(S) * ldo * 2);
  const dma_rsrc rl = dma_make_rsrc(lse, static_cast<int64_t>(S) * 4);
  const dma_rsrc rd = dma_make_rsrc(del, static_cast<int64_t>(S) * 4);
  const int lrow = grp * RPI + lane / LPR;                            // row of load 0
  const int lchk = ((lane % LPR) ^ qd_swz<DH>(lrow)) << 3;            // its logical column
  const uint32_t lq = static_cast<uint32_t>((lrow * ldq + lchk) * 2);
  const uint32_t lo = static_cast<uint32_t>((lrow * ldo + lchk) * 2);
  auto load_block = [&](int st, int qb) {
    if (!role_b) return;
    char* sb = ring + st * SB;
    const bool in = qb < S;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int p = grp + NG * i;
      const int64_t r = qb + static_cast<int64_t>(NG) * i * RPI;
      dma16(rq, sb + p * 1024, in ? lq + static_cast<uint32_t>(r * ldq * 2) : kDmaOob);
      dma16(ro, sb + BQ * DH * 2 + p * 1024, in ? lo + static_cast<uint32_t>(r * ldo * 2) : kDmaOob);
    }
    dma4(rl, sb + 4 * BQ * DH, in ? static_cast<uint32_t>((qb + lane) * 4) : kDmaOob);
    dma4(rd, sb + 4 * BQ * DH + 4 * BQ, in ? static_cast<uint32_t>((qb + lane) * 4) : kDmaOob);
  };

  // Per-lane LDS byte addresses, each set pointing into the stage of the
  // block it serves: plain reads (row cl, 16-byte chunk 2ks + hf) of Q
  // (wave A) or dO (wave B) for the score products, transposing reads (rows
  // tr_r and tr_r + 8) of dO (wave A) or Q (wave B) for the dV/dK products,
  // and the log-sum-exp (wave A) or delta (wave B) of the lane's first query.
  // The half, the 16-row groups and d blocks are immediates.
  uint32_t aq[N], at0[NDB], at1[NDB], al;
  {
    const uint32_t r0 = lds_addr(ring);
    const uint32_t plain = role_b ? 2u * BQ * DH : 0u, trans = role_b ? 0u : 2u * BQ * DH;
    const int sw_c = qd_swz<DH>(cl);
#pragma unroll
    for (int ks = 0; ks < N; ++ks) aq[ks] = r0 + plain + 2u * (cl * DH + (((2 * ks + hf) ^ sw_c) << 3));
    const int tr_r = 4 * hf + ((lane & 15) >> 2);
    const int tr_d = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
    const int sw0 = qd_swz<DH>(tr_r), sw1 = qd_swz<DH>(tr_r + 8);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d0 = db * 32 + tr_d;
      at0[db] = r0 + trans + 2u * (tr_r * DH + (((d0 >> 3) ^ sw0) << 3) + (d0 & 7));
      at1[db] = r0 + trans + 2u * ((tr_r + 8) * DH + (((d0 >> 3) ^ sw1) << 3) + (d0 & 7));
    }
    al = r0 + 4u * BQ * DH + (role_b ? 4u * BQ : 0u) + 16u * hf;
  }
  // the lane's 16-byte slots of the P exchange (floats 4c .. 4c+3 of its 16
  // at + 1024 c; parity 1 at + kDkPSlot)
  const uint32_t pslot = lds_addr(ring) + DK_NST * SB + grp * 4096 + 16u * lane;
  // moving a set from the stage of block b to that of block b + 1
  auto adv = [](int b) { return b % DK_NST == DK_NST - 1 ? static_cast<uint32_t>(-(DK_NST - 1) * SB) : static_cast<uint32_t>(SB); };
  auto move = [](auto& set, uint32_t d) {
#pragma unroll
    for (auto& x : set) x += d;
  };

  // Wave A, one half: S of half hs of the block aq points at, then the dV
  // product of half hv of the block at0/at1 point at (P of that half in pin)
  // with P of half hs (query block qb, for the mask and ALiBi) formed
  // between its MFMAs into pout and the exchange slot of parity par.
  auto half_a = [&](auto mask, auto do_s, auto do_v, int hs, int hv, int qb, int par, const bf16x8 (&pin)[2],
                    bf16x8 (&pout)[2]) {
    constexpr bool MASK = decltype(mask)::value, DS = decltype(do_s)::value, DV = decltype(do_v)::value;
    const uint32_t hq = 2u * hs * 32 * DH;
    floatx16 sc;
    struct Fr {
      bf16x8 q;
    };
    auto load = [&](Fr& f, int i) {
      if constexpr (DS) f.q = lds_frag(aq[i] + hq);
    };
    Fr fr[3];
    load(fr[0], 0);
    load(fr[1], 1);
    floatx4 l4[4];
    if constexpr (DS) {
#pragma unroll
      for (int g = 0; g < 4; ++g) l4[g] = lds_f4(al + 4u * (hs * 32 + 8 * g));
    }
    // S first (its fragments two steps ahead), the dV fragments meanwhile
    bf16x8 trf[N];
    auto load_tr = [&](int i) {
      if constexpr (DV) {
        const int db = i % NDB, c = i / NDB;
        const uint32_t rr = 2u * (hv * 32 + 16 * c) * DH;
        trf[i] = tr_pair(lds_tr(at0[db] + rr), lds_tr(at1[db] + rr));
      }
    };
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (i + 2 < N) load(fr[(i + 2) % 3], i + 2);
      load_tr(i);
      if constexpr (DS) sc = mfma(fr[i % 3].q, kv[i], i == 0 ? floatx16{} : sc);
      __builtin_amdgcn_sched_barrier(0);
    }
    const int t = key - (qb + hs * 32 + 4 * hf);  // key minus the lane's first query
    const float ab = al2 * static_cast<float>(t);  // ALiBi bias at that query
    floatx4 pf[4];  // P in float32 for B's dS
    auto softmax = [&](int v) {
      const int c = 8 * (v >> 2) + (v & 3);  // the element's query after the first
      float x = fmaf(sc[v], sl2, -l4[v >> 2][v & 3] * kLog2e);
      if constexpr (AL) x += fmaf(-al2, static_cast<float>(c), ab);
      float p = __builtin_amdgcn_exp2f(x);
      if constexpr (MASK) p = t > c ? 0.f : p;  // causal: keys after the query
      pout[v >> 3][v & 7] = static_cast<bf16>(p);
      pf[v >> 2][v & 3] = p;
    };
    // then the dV products with the softmax of S between them
    constexpr int EPI = 16 / N;  // softmax elements per dV MFMA
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if constexpr (DV) acc[i % NDB] = mfma(trf[i], pin[i / NDB], acc[i % NDB]);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (DS) {
#pragma unroll
        for (int e = 0; e < EPI; ++e) softmax(EPI * i + e);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (DS) {
#pragma unroll
      for (int g = 0; g < 4; ++g) lds_put(pslot + par * kDkPSlot + 1024u * g, pf[g]);
    }
  };
  // Wave B, one half: dP - delta of half hs of the block aq/al point at
  // into dpout, with dS of the previous half (P from the exchange slot of
  // parity par, dP - delta in dpin) formed between its MFMAs; then the dK
  // product of half hk of the block at0/at1 point at.
  auto half_b = [&](auto do_k, auto do_p, int hs, int hk, int par, const floatx16& dpin, floatx16& dpout) {
    constexpr bool DK = decltype(do_k)::value, DP = decltype(do_p)::value;
    const uint32_t hq = 2u * hs * 32 * DH;
    floatx4 pf[4];
    bf16x8 dsb[2];
    if constexpr (DK) {
#pragma unroll
      for (int g = 0; g < 4; ++g) pf[g] = lds_f4(pslot + par * kDkPSlot + 1024u * g);
    }
    floatx16 nd;
    if constexpr (DP) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const floatx4 t = lds_f4(al + 4u * (hs * 32 + 8 * g));
#pragma unroll
        for (int e = 0; e < 4; ++e) nd[4 * g + e] = t[e];
      }
    }
    bf16x8 of[3], trf[N];
    auto load = [&](int i) {
      if constexpr (DP) of[i % 3] = lds_frag(aq[i] + hq);
    };
    auto load_tr = [&](int i) {
      if constexpr (DK) {
        const int db = i % NDB, c = i / NDB;
        const uint32_t rr = 2u * (hk * 32 + 16 * c) * DH;
        trf[i] = tr_pair(lds_tr(at0[db] + rr), lds_tr(at1[db] + rr));
      }
    };
    auto ds = [&](int v) { dsb[v >> 3][v & 7] = static_cast<bf16>(pf[v >> 2][v & 3] * dpin[v]); };
    load(0);
    load(1);
    // dP (its fragments two steps ahead, the dK fragments meanwhile) with
    // dS of the previous half between its MFMAs; then the dK products
    constexpr int EPI = 16 / N;  // dS elements per dP MFMA
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (i + 2 < N) load(i + 2);
      load_tr(i);
      if constexpr (DP) dpout = mfma(of[i % 3], kv[i], i == 0 ? nd : dpout);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (DK) {
#pragma unroll
        for (int e = 0; e < EPI; ++e) ds(EPI * i + e);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (DK) {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        acc[i % NDB] = mfma(trf[i], dsb[i / NDB], acc[i % NDB]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  const std::integral_constant<bool, true> yes;
  const std::integral_constant<bool, false> no;
  const int q_first = k0;  // the first query that can see key k0
  const int nqb = (S - q_first) / BQ;
  // The whole walk for one role, so that the other role's state is not live
  // in it.
  auto walk = [&](auto is_b) {
    constexpr bool RB = decltype(is_b)::value;
    bf16x8 pbx[2], pby[2];  // wave A: P of the two halves of a block
    floatx16 dpx, dpy;      // wave B: dP - delta of the two halves of a block
    // one half: S/P or dP of half hs, the dV or dK product of half hv
    // (odd: the second half of a block; A writes the P slot of its parity,
    // B reads the other)
    auto half = [&](auto mask, auto first, auto second, int hs, int hv, int qb, bool odd) {
      if constexpr (!RB) {
        if (odd)
          half_a(mask, first, second, hs, hv, qb, 1, pbx, pby);
        else
          half_a(mask, first, second, hs, hv, qb, 0, pby, pbx);
      } else {
        // B: first = the dK product (of the previous half), second = dP
        if (odd)
          half_b(first, second, hs, hv, 0, dpx, dpy);
        else
          half_b(first, second, hs, hv, 1, dpy, dpx);
      }
    };
    // Block 0 into the ring and the K/V fragments (1 in flight), then its
    // first half.
    load_block(0, q_first);
    load_kv();
    load_block(1, q_first + BQ);
    dma_barrier<NL>();  // block 0 has landed
    if constexpr (!RB)
      half(yes, yes, no, 0, 0, q_first, false);
    else
      half(yes, no, yes, 0, 0, q_first, false);
    lds_barrier();
    load_block(2, q_first + 2 * BQ);
    // its second half, with the products of the first
    half(yes, yes, yes, 1, 0, q_first, true);
    dma_barrier<NL>();  // block 1 has landed
    move(aq, adv(0));
    al += adv(0);
    // Block j: first half (with the products of block j-1's second half);
    // barrier; block j+2 goes to the stage block j-1 left; second half (with
    // the products of the first); barrier (block j+1 has landed).
    auto block = [&](auto mask, int j) {
      const int qb = q_first + j * BQ;
      half(mask, yes, yes, 0, 1, qb, false);
      lds_barrier();
      load_block((j + 2) % DK_NST, qb + 2 * BQ);
      move(at0, adv(j - 1));
      move(at1, adv(j - 1));
      half(mask, yes, yes, 1, 0, qb, true);
      dma_barrier<NL>();
      move(aq, adv(j));
      al += adv(j);
    };
    // Only the blocks that start before the workgroup's last key hold
    // queries that some of its keys come after.
    constexpr int kMaskBlocks = BKEYS / BQ;
    int j = 1;
    for (; j < nqb && j < kMaskBlocks; ++j) block(yes, j);
    for (; j < nqb; ++j) block(no, j);
    // the products of the last half
    if constexpr (!RB)
      half(no, no, yes, 0, 1, 0, false);
    else
      half(no, yes, no, 0, 1, 0, false);
  };
  if (role_b)
    walk(yes);
  else
    walk(no);
  dma_barrier<0>();  // no load may still write LDS when the workgroup ends
  if (active && key < S) {
    bf16* G = static_cast<bf16*>(a.out) + (static_cast<int64_t>(seq) * S + key) * ldq + head * DH +
              (role_b ? 1ll : 2ll) * H * DH;
    const float f = role_b ? a.scale : 1.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        __attribute__((aligned(8))) bf16 t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) t[i] = static_cast<bf16>(acc[db][4 * g + i] * f);
        *reinterpret_cast<uint2*>(G + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(t);
      }
  }
}

// Forward.  A workgroup owns 256 query rows; each wave owns RPW of them as
// RPW/32 MFMA blocks that share every K and V fragment it reads from LDS.
// K/V blocks of 64 keys go from global memory straight into a four-stage LDS
// ring ([key][d], as in the dQ kernel), so a block's loads have two
// block-times to land; V^T comes from transposing reads of the [key][d]
// block in the accumulator's key permutation.  Online softmax in base 2 with
// lazy rescaling; causal mask on diagonal blocks only.
// AL: add the ALiBi bias to the scaled scores (in log2 units: slope * log2e
// per position of distance).
template <int DH>
constexpr int fwd_stage_bytes() { return 4 * FKV * DH; }  // K block, then V block
constexpr int FWD_NST = 4;

template <int DH, int RPW, bool AL>
__global__ __launch_bounds__(64 * (FWQ / RPW)) void ld_attn_fwd_bf16(AttnArgs a) {
  constexpr int NSB = RPW / 32, NW = FWQ / RPW, SB = fwd_stage_bytes<DH>();
  constexpr int RPI = 512 / DH, LPR = 64 / RPI;   // rows per 1 KB load, lanes per row
  constexpr int NPW = (FKV * DH * 2 / 1024) / NW;  // 1 KB loads per wave per tensor and block
  constexpr int NL = 2 * NPW;
  static_assert(NPW >= 1, "every wave loads part of each block");
  extern __shared__ __align__(16) char ring[];
  const int S = a.S, H = a.H;
  const int n_qt = (S + FWQ - 1) / FWQ;
  // grid (head, sequence, tile): the tile index varies slowest, so every
  // (heaviest) last query tile is dispatched before any lighter one
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.z);
  const int head = blockIdx.x, seq = blockIdx.y;
  if (seq >= seq_count(a)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hf = lane >> 5, cl = lane & 31;
  const int q0 = qt * FWQ, qw = q0 + wave * RPW;
  const int64_t ldq = 3ll * H * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  const bf16* Kp = base + static_cast<int64_t>(H) * DH + head * DH;
  const bf16* Vp = base + 2ll * H * DH + head * DH;
  const float sl2 = a.scale * kLog2e;
  const float al2 = AL ? alibi_slope(head, H) * kLog2e : 0.f;

  bf16x8 qf[NSB][DH / 16];
  floatx16 o[NSB][DH / 32];
  float m[NSB], l[NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int qrow = qw + sb * 32 + cl;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks)
      qf[sb][ks] = qrow < S ? load8(Qp + static_cast<int64_t>(qrow) * ldq + ks * 16 + hf * 8) : zero8();
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[sb][db][v] = 0.f;
    m[sb] = -INFINITY;
    l[sb] = 0.f;
  }
  // The fragments must have arrived before the first LDS load is issued
  // (the compiler does not see those loads).
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) asm volatile("" ::"v"(qf[sb][ks]));

  // Loads of key block k0 into stage st; blocks at or past the end read zeros.
  const dma_rsrc rk = dma_make_rsrc(Kp, static_cast<int64_t>(S) * ldq * 2);
  const dma_rsrc rv = dma_make_rsrc(Vp, static_cast<int64_t>(S) * ldq * 2);
  const int lrow = wave * RPI + lane / LPR;
  const int lchk = ((lane % LPR) ^ qd_swz<DH>(lrow)) << 3;
  const uint32_t lk = static_cast<uint32_t>((lrow * ldq + lchk) * 2);
  auto load_block = [&](int st, int k0) {
    char* sbp = ring + st * SB;
    const bool in = k0 < S;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int p = wave + NW * i;
      const uint32_t r = static_cast<uint32_t>((static_cast<int64_t>(k0) + NW * i * RPI) * ldq * 2);
      dma16(rk, sbp + p * 1024, in ? lk + r : kDmaOob);
      dma16(rv, sbp + FKV * DH * 2 + p * 1024, in ? lk + r : kDmaOob);
    }
  };
  // Per-lane LDS byte addresses in the stage of the current block: plain
  // reads of K (row cl, 16-byte chunk 2ks + hf) and transposing reads of V
  // (rows tr_r and tr_r + 8).
  uint32_t ak[DH / 16], at0[DH / 32], at1[DH / 32];
  {
    const uint32_t r0 = lds_addr(ring);
    const int sw_c = qd_swz<DH>(cl);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) ak[ks] = r0 + 2u * (cl * DH + (((2 * ks + hf) ^ sw_c) << 3));
    const int tr_r = 4 * hf + ((lane & 15) >> 2);
    const int tr_d = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
    const int sw0 = qd_swz<DH>(tr_r), sw1 = qd_swz<DH>(tr_r + 8);
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) {
      const int d0 = db * 32 + tr_d;
      at0[db] = r0 + 2u * FKV * DH + 2u * (tr_r * DH + (((d0 >> 3) ^ sw0) << 3) + (d0 & 7));
      at1[db] = r0 + 2u * FKV * DH + 2u * ((tr_r + 8) * DH + (((d0 >> 3) ^ sw1) << 3) + (d0 & 7));
    }
  }

  const int kv_end = min(S, q0 + FWQ);
  const int nkb = (kv_end + FKV - 1) / FKV;
  load_block(0, 0);
  load_block(1, FKV);
  load_block(2, 2 * FKV);
  for (int kb = 0; kb < nkb; ++kb) {
    const int k0 = kb * FKV, st = kb & (FWD_NST - 1);
    // block kb has landed (blocks kb+1, kb+2 may be in flight); the stage of
    // block kb-1 is no longer read and takes block kb+3
    dma_barrier<2 * NL>();
    load_block((kb + 3) & (FWD_NST - 1), k0 + 3 * FKV);
    if (qw < S && k0 <= qw + RPW - 1) {
      const bool diag = k0 + FKV - 1 > qw;  // some key of the block is past some row
      // scores of every 32-row block: each K fragment feeds NSB MFMA chains;
      // fragments read two steps ahead (step i: ks = i / 2, kh = i % 2)
      constexpr int NS = 2 * (DH / 16), NP = 4 * (DH / 32);
      floatx16 sc[NSB][2];
      bf16x8 kfr[3];
      auto ldk = [&](int i) { kfr[i % 3] = lds_frag(ak[i / 2] + 2u * (i % 2) * 32 * DH); };
      ldk(0);
      ldk(1);
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        if (i + 2 < NS) ldk(i + 2);
        const int ks = i / 2, kh = i % 2;
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) sc[sb][kh] = mfma(kfr[i % 3], qf[sb][ks], ks == 0 ? floatx16{} : sc[sb][kh]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // the first V^T fragments land during the softmax (step i: kh = i /
      // (2 NDB), c = i / NDB % 2, db = i % NDB)
      bf16x8 vfr[3];
      auto ldv = [&](int i) {
        const int kh = i / (2 * (DH / 32)), c = (i / (DH / 32)) % 2, db = i % (DH / 32);
        const uint32_t rr = 2u * (kh * 32 + 16 * c) * DH;
        vfr[i % 3] = tr_pair(lds_tr(at0[db] + rr), lds_tr(at1[db] + rr));
      };
      ldv(0);
      ldv(1);
      bf16x8 pb[NSB][2][2];
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb) {
        const int qrow = qw + sb * 32 + cl;
        const float ab = al2 * static_cast<float>(k0 + 4 * hf - qrow);  // bias of the lane's first key
        float mx = -INFINITY;
        // With ALiBi the scores are scaled and biased here; without, they
        // stay raw until the exponent (scale > 0, so the maximum of the raw
        // scores times the scale is the maximum of the scaled ones).
        if constexpr (AL) {
#pragma unroll
          for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int v = 0; v < 16; ++v)
              sc[sb][kh][v] = fmaf(sc[sb][kh][v], sl2, fmaf(al2, static_cast<float>(kh * 32 + 8 * (v >> 2) + (v & 3)), ab));
        }
        if (diag) {  // causal mask, only on blocks that reach past a row (wave-uniform)
          const int t = qrow - k0 - 4 * hf;  // the row minus the lane's first key
#pragma unroll
          for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int v = 0; v < 16; ++v)
              if (kh * 32 + 8 * (v >> 2) + (v & 3) > t) sc[sb][kh][v] = -INFINITY;
        }
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[sb][kh][v]);
        mx = half_max(mx);
        if constexpr (!AL) mx *= sl2;
        // Lazy rescaling: the running maximum only moves (and O, l are only
        // rescaled) when a row's maximum grows by more than 8 in log2 units;
        // otherwise p = 2^(s - m) stays below 2^8, exact enough in bf16 and
        // far from float overflow, and the result O / l is unchanged.
        const bool grow = mx > m[sb] + 8.f;
        if (__builtin_amdgcn_read_exec() & __ballot(grow)) {
          const float m_new = grow ? mx : m[sb];
          const float alpha = __builtin_amdgcn_exp2f(m[sb] - m_new);
          m[sb] = m_new;
          l[sb] *= alpha;
#pragma unroll
          for (int db = 0; db < DH / 32; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[sb][db][v] *= alpha;
        }
        float ls = 0.f;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float p = __builtin_amdgcn_exp2f(AL ? sc[sb][kh][v] - m[sb] : fmaf(sc[sb][kh][v], sl2, -m[sb]));
            ls += p;
            pb[sb][kh][v >> 3][v & 7] = static_cast<bf16>(p);
          }
        l[sb] += ls;
      }
      // O^T += V^T P^T; consecutive MFMAs go to different accumulators (the
      // d blocks innermost), so none waits on the one before it
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        if (i + 2 < NP) ldv(i + 2);
        const int kh = i / (2 * (DH / 32)), c = (i / (DH / 32)) % 2, db = i % (DH / 32);
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) o[sb][db] = mfma(vfr[i % 3], pb[sb][kh][c], o[sb][db]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // next block: one stage on (wrapping around the ring)
    const uint32_t adv = st == FWD_NST - 1 ? static_cast<uint32_t>(-(FWD_NST - 1) * SB) : static_cast<uint32_t>(SB);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) ak[ks] += adv;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) {
      at0[db] += adv;
      at1[db] += adv;
    }
  }
  dma_barrier<0>();  // no load may still write LDS when the workgroup ends
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int qrow = qw + sb * 32 + cl;
    const float lt = half_sum(l[sb]);
    if (qrow < S) {
      const float inv = 1.f / lt;
      bf16* Op = static_cast<bf16*>(a.out) + (static_cast<int64_t>(seq) * S + qrow) * (static_cast<int64_t>(H) * DH) + head * DH;
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          __attribute__((aligned(8))) bf16 t[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) t[i] = static_cast<bf16>(o[sb][db][4 * g + i] * inv);
          *reinterpret_cast<uint2*>(Op + db * 32 + 8 * g + 4 * hf) = *reinterpret_cast<uint2*>(t);
        }
      if (hf == 0) a.lse[(static_cast<int64_t>(seq) * H + head) * S + qrow] = (m[sb] + log2f(lt)) * kLn2;
    }
  }
}

template <int DH>
constexpr size_t dkdv_lds_bytes() {
  return static_cast<size_t>(DK_NST) * dk_stage_bytes<DH>() + kDkPBytes;
}
static_assert(dkdv_lds_bytes<128>() <= 160 * 1024, "the dK/dV ring and P area fit the LDS");

constexpr int DQ_ROWS = 256;  // query rows per dQ workgroup (8 waves x 32)

// dQ.  A workgroup of 8 waves owns 256 query rows (32 per wave, two waves per
// SIMD) and walks the 64-key blocks up to the diagonal.  K and V blocks go
// from global memory straight into a four-stage LDS ring ([key][d] without
// padding, 16-byte chunks XOR-swizzled by the key as in the dK/dV ring), so a
// block's loads have two block-times to land.  Scores are formed transposed
// (S^T = K Q^T), so the query's log-sum-exp and delta are per lane, and
// dS^T feeds dQ^T += K^T dS^T directly, K^T coming from the same [key][d]
// block through transposing reads in the accumulator's key permutation.
// Fragment addresses are per-lane offsets moved by one stage per block; the
// causal mask is applied on diagonal blocks only.
constexpr int DQ_NST = 4;
template <int DH>
constexpr int dq_stage_bytes() { return 4 * FKV * DH; }  // K block, then V block

template <int DH, bool AL>
__global__ __launch_bounds__(512) void ld_attn_bwd_dq_bf16(AttnArgs a) {
  constexpr int NW = 8, SB = dq_stage_bytes<DH>();
  constexpr int RPI = 512 / DH, LPR = 64 / RPI;   // rows per 1 KB load, lanes per row
  constexpr int NPW = (FKV * DH * 2 / 1024) / NW;  // 1 KB loads per wave per tensor and block
  constexpr int NL = 2 * NPW;                      // loads per wave per block
  static_assert(NPW >= 1, "every wave loads part of each block");
  extern __shared__ __align__(16) char ring[];
  const int S = a.S, H = a.H;
  const int n_qt = (S + DQ_ROWS - 1) / DQ_ROWS;
  // grid (head, sequence, tile), tile slowest: heavy (late) query tiles first
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.z);
  const int head = blockIdx.x, seq = blockIdx.y;
  if (seq >= seq_count(a)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hf = lane >> 5, cl = lane & 31;
  const int q0 = qt * DQ_ROWS, qw = q0 + wave * 32, qrow = qw + cl;
  const int64_t ldq = 3ll * H * DH, ldo = static_cast<int64_t>(H) * DH;
  const bf16* base = static_cast<const bf16*>(a.qkv) + static_cast<int64_t>(seq) * S * ldq;
  const bf16* Qp = base + head * DH;
  const bf16* Kp = base + static_cast<int64_t>(H) * DH + head * DH;
  const bf16* Vp = base + 2ll * H * DH + head * DH;
  const bf16* dOp = static_cast<const bf16*>(a.go) + static_cast<int64_t>(seq) * S * ldo + head * DH;
  const float sl2 = a.scale * kLog2e;
  const float al2 = AL ? alibi_slope(head, H) * kLog2e : 0.f;

  const bool qok = qrow < S;
  const int64_t srow = (static_cast<int64_t>(seq) * H + head) * S + (qok ? qrow : 0);
  const float lse2 = qok ? a.lse[srow] * kLog2e : 0.f;
  bf16x8 qf[DH / 16], of[DH / 16];
  const bf16* Orow = static_cast<const bf16*>(a.o) + static_cast<int64_t>(seq) * S * ldo + head * DH +
                     static_cast<int64_t>(qok ? qrow : 0) * ldo;
  float dsum = 0.f;
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) {
    qf[ks] = qok ? load8(Qp + static_cast<int64_t>(qrow) * ldq + ks * 16 + hf * 8) : zero8();
    of[ks] = qok ? load8(dOp + static_cast<int64_t>(qrow) * ldo + ks * 16 + hf * 8) : zero8();
    const bf16x8 ov = qok ? load8(Orow + ks * 16 + hf * 8) : zero8();
#pragma unroll
    for (int e = 0; e < 8; ++e) dsum = fmaf(static_cast<float>(of[ks][e]), static_cast<float>(ov[e]), dsum);
  }
  // delta of the row (the two half-waves hold its two halves of d), stored
  // negated for the dK/dV kernel, which runs after this one
  const float dl = -half_sum(dsum);
  if (qok && hf == 0) a.delta[srow] = dl;
  // the store has completed before the first LDS load is issued: those are
  // counted by the waits below, which know of no other memory operation
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // The fragments must have arrived before the first LDS load is issued
  // (the compiler does not see those loads).
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) asm volatile("" ::"v"(qf[ks]), "v"(of[ks]));
  asm volatile("" ::"v"(lse2), "v"(dl));
  floatx16 dq[DH / 32];
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) dq[db][v] = 0.f;
  // dP accumulations start from the row's negated delta: the MFMAs give dP -
  // delta
  floatx16 dls;
#pragma unroll
  for (int v = 0; v < 16; ++v) dls[v] = dl;

  // Loads of key block k0 into stage st; blocks at or past the end read zeros.
  const dma_rsrc rk = dma_make_rsrc(Kp, static_cast<int64_t>(S) * ldq * 2);
  const dma_rsrc rv = dma_make_rsrc(Vp, static_cast<int64_t>(S) * ldq * 2);
  const int lrow = wave * RPI + lane / LPR;
  const int lchk = ((lane % LPR) ^ qd_swz<DH>(lrow)) << 3;
  const uint32_t lk = static_cast<uint32_t>((lrow * ldq + lchk) * 2);
  auto load_block = [&](int st, int k0) {
    char* sb = ring + st * SB;
    const bool in = k0 < S;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int p = wave + NW * i;
      const uint32_t r = static_cast<uint32_t>((static_cast<int64_t>(k0) + NW * i * RPI) * ldq * 2);
      dma16(rk, sb + p * 1024, in ? lk + r : kDmaOob);
      dma16(rv, sb + FKV * DH * 2 + p * 1024, in ? lk + r : kDmaOob);
    }
  };
  // Per-lane LDS byte addresses in the stage of the current block: plain
  // reads of K (row cl, 16-byte chunk 2ks + hf; V one block further) and the
  // transposing reads of K (rows tr_r and tr_r + 8).
  uint32_t ak[DH / 16], at0[DH / 32], at1[DH / 32];
  {
    const uint32_t r0 = lds_addr(ring);
    const int sw_c = qd_swz<DH>(cl);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) ak[ks] = r0 + 2u * (cl * DH + (((2 * ks + hf) ^ sw_c) << 3));
    const int tr_r = 4 * hf + ((lane & 15) >> 2);
    const int tr_d = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
    const int sw0 = qd_swz<DH>(tr_r), sw1 = qd_swz<DH>(tr_r + 8);
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) {
      const int d0 = db * 32 + tr_d;
      at0[db] = r0 + 2u * (tr_r * DH + (((d0 >> 3) ^ sw0) << 3) + (d0 & 7));
      at1[db] = r0 + 2u * ((tr_r + 8) * DH + (((d0 >> 3) ^ sw1) << 3) + (d0 & 7));
    }
  }
  constexpr uint32_t kVb = 2u * FKV * DH;  // V block after the K block (bytes)

  const int kv_end = min(S, q0 + DQ_ROWS);
  const int nkb = kv_end / FKV;
  load_block(0, 0);
  load_block(1, FKV);
  load_block(2, 2 * FKV);
  for (int kb = 0; kb < nkb; ++kb) {
    const int k0 = kb * FKV, st = kb & (DQ_NST - 1);
    // block kb has landed (blocks kb+1, kb+2 may be in flight); the stage of
    // block kb-1 is no longer read and takes block kb+3
    dma_barrier<2 * NL>();
    load_block((kb + 3) & (DQ_NST - 1), k0 + 3 * FKV);
    if (qw < S && k0 <= qw + 31) {
      const bool diag = k0 + FKV - 1 > qw;  // some key of the block is past some row
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        constexpr int N = DH / 16, NC = 2 * (DH / 32);
        const uint32_t hk = 2u * kh * 32 * DH;
        // S^T and dP^T - delta, the K and V fragments read two steps ahead
        bf16x8 kfr[3], vfr[3];
        auto ld = [&](int ks) {
          kfr[ks % 3] = lds_frag(ak[ks] + hk);
          vfr[ks % 3] = lds_frag(ak[ks] + hk + kVb);
        };
        ld(0);
        ld(1);
        floatx16 st_, dpt;
#pragma unroll
        for (int ks = 0; ks < N; ++ks) {
          if (ks + 2 < N) ld(ks + 2);
          st_ = mfma(kfr[ks % 3], qf[ks], ks == 0 ? floatx16{} : st_);
          dpt = mfma(vfr[ks % 3], of[ks], ks == 0 ? dls : dpt);
          __builtin_amdgcn_sched_barrier(0);
        }
        // the first K^T fragments of the dQ product land during the softmax
        bf16x8 tf[3];
        auto ldt = [&](int i) {
          const int db = i % (DH / 32), c = i / (DH / 32);
          const uint32_t rr = hk + 2u * 16 * c * DH;
          tf[i % 3] = tr_pair(lds_tr(at0[db] + rr), lds_tr(at1[db] + rr));
        };
        ldt(0);
        ldt(1);
        bf16x8 dsb[2];
        const float ab = al2 * static_cast<float>(k0 + kh * 32 + 4 * hf - qrow);  // bias of the lane's first key
        float pv[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = fmaf(st_[v], sl2, -lse2);
          if constexpr (AL) x += fmaf(al2, static_cast<float>(8 * (v >> 2) + (v & 3)), ab);
          pv[v] = __builtin_amdgcn_exp2f(x);
        }
        if (diag) {  // causal mask (wave-uniform branch): keys after the row
          const int t = qrow - (k0 + kh * 32 + 4 * hf);  // the row minus the lane's first key
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (8 * (v >> 2) + (v & 3) > t) pv[v] = 0.f;
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) dsb[v >> 3][v & 7] = static_cast<bf16>(pv[v] * dpt[v]);
        // dQ^T += K^T dS^T, the d blocks innermost (consecutive MFMAs use
        // different accumulators), fragments two steps ahead
#pragma unroll
        for (int i = 0; i < NC; ++i) {
          if (i + 2 < NC) ldt(i + 2);
          dq[i % (DH / 32)] = mfma(tf[i % 3], dsb[i / (DH / 32)], dq[i % (DH / 32)]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    // next block: one stage on (wrapping around the ring)
    const uint32_t adv = st == DQ_NST - 1 ? static_cast<uint32_t>(-(DQ_NST - 1) * SB) : static_cast<uint32_t>(SB);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) ak[ks] += adv;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) {
      at0[db] += adv;
      at1[db] += adv;
    }
  }
  dma_barrier<0>();  // no load may still write LDS when the workgroup ends
  if (qok) {
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

template <int DH>
constexpr size_t dq_lds_bytes() {
  return static_cast<size_t>(DQ_NST) * dq_stage_bytes<DH>();
}

// ------------------------------------------------------------ fp32 (SIMT)

constexpr int ST = 64;  // rows per workgroup and keys per LDS tile

template <int DH>
__global__ __launch_bounds__(64) void ld_attn_fwd_f32(AttnArgs a) {
  __shared__ float Ks[ST][DH], Vs[ST][DH];
  const int S = a.S, H = a.H;
  const int head = blockIdx.y, seq = blockIdx.z;
  const float al = a.alibi ? alibi_slope(head, H) : 0.f;  // ALiBi slope (natural units)
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
      s = s * a.scale - al * static_cast<float>(q - key);
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
  const float al = a.alibi ? alibi_slope(head, H) : 0.f;  // ALiBi slope (natural units)
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
      const float p = expf(s * a.scale - al * static_cast<float>(q - key) - lse);
      const float ds = p * (dp + dl);
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
  const float al = a.alibi ? alibi_slope(head, H) : 0.f;  // ALiBi slope (natural units)
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
        const float p = expf(s * a.scale - al * static_cast<float>(q - key) - ls[j]);
        const float ds = p * (dp + dls[j]);
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
      const dim3 grid(a.H, a.n_seq, (a.S + FWQ - 1) / FWQ);
      constexpr int rpw = kFwdRowsPerWave;
      if (a.alibi)
        hipLaunchKernelGGL((ld_attn_fwd_bf16<DH, rpw, true>), grid, dim3(64 * (FWQ / rpw)),
                           FWD_NST * fwd_stage_bytes<DH>(), s, a);
      else
        hipLaunchKernelGGL((ld_attn_fwd_bf16<DH, rpw, false>), grid, dim3(64 * (FWQ / rpw)),
                           FWD_NST * fwd_stage_bytes<DH>(), s, a);
      return hipGetLastError();
    }
  }
  if constexpr (DH <= 64) {
    const dim3 grid((a.S + ST - 1) / ST, a.H, a.n_seq);
    hipLaunchKernelGGL(ld_attn_fwd_f32<DH>, grid, dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

// bf16: part 0 is the dQ kernel (it also forms and stores delta), part 1
// the dK/dV kernel; float32: delta, dK/dV, dQ.
template <int DH>
hipError_t bwd_dh(int dtype, int part, const AttnArgs& a, hipStream_t s) {
  const int64_t tokens = static_cast<int64_t>(a.n_seq) * a.S;  // one wave per token
  const dim3 dgrid(static_cast<unsigned>((tokens + 3) / 4));
  if constexpr (DH >= 64) {
    if (dtype == LD_BF16) {
      if (part == 1) {
        constexpr int ng = DK_GROUPS;
        const dim3 grid(a.H, a.n_seq, (a.S + 32 * ng - 1) / (32 * ng));
        if (a.alibi)
          hipLaunchKernelGGL((ld_attn_bwd_dkdv_bf16<DH, ng, true>), grid, dim3(128 * ng), dkdv_lds_bytes<DH>(), s, a);
        else
          hipLaunchKernelGGL((ld_attn_bwd_dkdv_bf16<DH, ng, false>), grid, dim3(128 * ng), dkdv_lds_bytes<DH>(), s, a);
      } else if (part == 0) {
        const dim3 grid(a.H, a.n_seq, (a.S + DQ_ROWS - 1) / DQ_ROWS);
        if (a.alibi)
          hipLaunchKernelGGL((ld_attn_bwd_dq_bf16<DH, true>), grid, dim3(512), dq_lds_bytes<DH>(), s, a);
        else
          hipLaunchKernelGGL((ld_attn_bwd_dq_bf16<DH, false>), grid, dim3(512), dq_lds_bytes<DH>(), s, a);
      }
      return hipGetLastError();
    }
  }
  if constexpr (DH <= 64) {
    const dim3 grid((a.S + ST - 1) / ST, a.H, a.n_seq);
    if (part == 0)
      hipLaunchKernelGGL((ld_attn_delta<float, DH>), dgrid, dim3(256), 0, s, a);
    else if (part == 1)
      hipLaunchKernelGGL(ld_attn_bwd_dkdv_f32<DH>, grid, dim3(64), 0, s, a);
    else
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

int attn_bwd_parts(int dtype) { return dtype == LD_BF16 ? 2 : 3; }

const char* attn_bwd_kernel_name(int dtype, int part) {
  static const char* names[2][3] = {{"ld_attn_delta", "ld_attn_bwd_dkdv_f32", "ld_attn_bwd_dq_f32"},
                                    {"ld_attn_bwd_dq_bf16", "ld_attn_bwd_dkdv_bf16", ""}};
  return names[dtype == LD_BF16 ? 1 : 0][part];
}

hipError_t launch_attn_bwd_part(int dtype, int part, const AttnArgs& a, hipStream_t s) {
  if (a.n_seq <= 0) return hipSuccess;
  if (dtype == LD_BF16) {
    if (a.dh == 64) return bwd_dh<64>(dtype, part, a, s);
    if (a.dh == 128) return bwd_dh<128>(dtype, part, a, s);
    return hipErrorInvalidValue;
  }
  switch (a.dh) {
    case 16: return bwd_dh<16>(dtype, part, a, s);
    case 32: return bwd_dh<32>(dtype, part, a, s);
    case 64: return bwd_dh<64>(dtype, part, a, s);
  }
  return hipErrorInvalidValue;
}

// ----------------------------------------------- fixed scratch, no allocation
// The backward's only scratch is delta = rowsum(dO * O).  The no-allocation
// entry point keeps it in this array instead of a caller workspace; each GPU
// holds its own copy until the process ends, and every call on a GPU shares
// it (calls that overlap on one GPU race).  The kernel that forms delta (dQ
// in bf16, a delta kernel in float32) writes every entry the dK/dV kernel
// reads before it runs, so nothing needs clearing.  On the host
// the array's name is only a stand-in: kernels get the address
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[kAttnScratchBytes / sizeof(float)];

constexpr int kScratchMaxDevices = 64;

hipError_t attn_scratch_ptr(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchMaxDevices) return hipErrorInvalidDevice;
  static std::mutex mu;
  static void* addr[kScratchMaxDevices] = {};
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = static_cast<float*>(addr[dev]);
  return hipSuccess;
}

hipError_t launch_attn_bwd(int dtype, const AttnArgs& a, hipStream_t s) {
  for (int part = 0; part < attn_bwd_parts(dtype); ++part) {
    const hipError_t e = launch_attn_bwd_part(dtype, part, a, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ld

// Internal declarations shared by the HIP kernel translation units and the
// host-side C ABI.  Not installed; the public surface is include/layerdrop.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layerdrop.h"

namespace ld {

using bf16 = __bf16;

// ------------------------------------------------ global-to-LDS loads
// Buffer loads with an LDS destination: each lane's data goes to LDS at a
// wave-uniform base plus (bytes per lane) * lane, so the layout in LDS is set
// by which global address each lane fetches.  A raw buffer descriptor bounds
// them: offsets at or past its size (kDmaOob is past every size used) return
// zeros.  They are issued as inline assembly, so the compiler does not track
// them: code that issues them waits itself (s_waitcnt vmcnt) before reading
// what they wrote, and issues no compiler-visible global loads whose waits
// would be miscounted meanwhile.  No other code in the kernels that use them
// reads m0.

typedef int dma_rsrc __attribute__((ext_vector_type(4)));
constexpr uint32_t kDmaOob = 0x80000000u;
constexpr int64_t kDmaMaxSpan = 0x7FFFFFFFll;  // bytes one descriptor may cover

__device__ __forceinline__ dma_rsrc dma_make_rsrc(const void* base, int64_t bytes) {
  const int64_t n = bytes < 0 ? 0 : (bytes > kDmaMaxSpan ? kDmaMaxSpan : bytes);
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return dma_rsrc{static_cast<int>(static_cast<uint32_t>(a)), static_cast<int>((a >> 32) & 0xFFFF),
                  static_cast<int>(n), 0x00020000};
}

// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)(p)));
}

// 16 bytes per lane from buffer offset `voff` to LDS `lds` + 16 * lane.
__device__ __forceinline__ void dma16(dma_rsrc rs, const void* lds, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds_addr(lds)),
               "v"(voff), "s"(rs));
}

// 4 bytes per lane from buffer offset `voff` to LDS `lds` + 4 * lane.
__device__ __forceinline__ void dma4(dma_rsrc rs, const void* lds, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds" ::"s"(lds_addr(lds)),
               "v"(voff), "s"(rs));
}

// Waits until at most N of this wave's vector memory operations are in
// flight and its LDS accesses are done, then meets the workgroup.  A
// compiler barrier for memory.
template <int N>
__device__ __forceinline__ void dma_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// ---------------------------------------------------------------- SwiGLU
// SwiGLU on float inputs (the gate u and up v as stored): s = silu(u) v, and
// the gradients gu = g v silu'(u), gv = g silu(u) with
// silu'(u) = sigmoid(u) (1 + u (1 - sigmoid(u))).  One definition for the
// elementwise kernels and the GEMM epilogues that fuse them; the fused ones
// apply it to float32 accumulator values where the elementwise kernels read
// the stored bf16 tensors.
// sigmoid(u) = 1 / (1 + 2^(-u log2 e)) with the hardware base-2 exponential
// and reciprocal (v_exp_f32, v_rcp_f32, about 1 ulp each): two instructions
// where expf and a correctly rounded division take a range reduction and a
// division sequence; far below the bf16 rounding the outputs take.  u = -inf
// gives 0, u = +inf gives 1.
__device__ __forceinline__ float swiglu_sigmoid(float u) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(u * -1.4426950408889634f));
}
__device__ __forceinline__ float swiglu_fwd_f(float u, float v) { return u * swiglu_sigmoid(u) * v; }
__device__ __forceinline__ void swiglu_bwd_f(float u, float v, float g, float& gu, float& gv) {
  const float sg = swiglu_sigmoid(u);
  gu = g * v * sg * (1.f + u * (1.f - sg));
  gv = g * u * sg;
}

// ------------------------------------------------------------ kernel args

// Rows of a compacted activation block.  When dev_count is set the row count
// is (*dev_count) * mult, read on the device, so no host sync is needed on the
// kept count; otherwise it is `rows`.
struct RowCount {
  const int32_t* dev_count;
  int32_t mult;
  int64_t rows;
};

// Mapping from a compacted row m to a row of a [B, S, d] tensor:
// row(m) = idx[m / S] * S + m % S, or m itself when idx is null.
struct RowMap {
  const int32_t* idx;
  int32_t S;
};

// ------------------------------------------------------ Philox4x64-10
// Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3"
// (SC'11): 10 rounds of two 64x64->128 multiplies, the key bumped by the
// Weyl constants between rounds.  Host and device share this definition, so
// the host can take the per-batch draws itself.
struct Philox4 {
  uint64_t w[4];
};

__host__ __device__ inline uint64_t mulhi64(uint64_t a, uint64_t b) {
  return static_cast<uint64_t>((static_cast<unsigned __int128>(a) * b) >> 64);
}

__host__ __device__ inline Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                 uint64_t k0, uint64_t k1) {
  constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;
  constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint64_t lo0 = kM0 * c0, hi0 = mulhi64(kM0, c0);
    const uint64_t lo1 = kM1 * c2, hi1 = mulhi64(kM1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0;
    const uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Philox4{{c0, c1, c2, c3}};
}

// The Bernoulli draws of the masks.  Per sequence: block (b, l, t, 0); per
// batch: block (0, l, t, 1); key (seed, 0).  Mask m of a layer (0: attention
// or whole layer, 1: FFN under sub-layer granularity) takes word m.
__host__ __device__ inline uint64_t mask_draw(uint64_t b, uint64_t layer, uint64_t step, uint64_t seed,
                                              int per_batch, int m) {
  const Philox4 r = philox4x64_10(per_batch ? 0 : b, layer, step, per_batch ? 1 : 0, seed, 0);
  return r.w[m];
}

constexpr int kMaxMaskLayers = 128;

struct MaskArgs {
  uint64_t thr[kMaxMaskLayers];     // drop iff word < thr (when !drop_all)
  uint8_t drop_all[kMaxMaskLayers]; // p >= 1
  float r[kMaxMaskLayers];          // residual scale per layer (0 for p >= 1)
  int32_t n_layers, batch, first_layer;
  int32_t n_masks;                  // 1, or 2 under sub-layer granularity
  int32_t per_batch;                // one draw per (layer, step) for the batch
  uint64_t seed, step;
  const uint8_t* keep_override;     // [n_layers][n_masks][batch] or null
  uint8_t* keep;                    // [n_layers][n_masks][batch]
  int32_t* idx;                     // [n_layers][n_masks][batch]
  int32_t* count;                   // [n_layers][n_masks]
  float* r_out;                     // [n_layers] or null: copy of r for the layer
};

// Zero fill of up to 6 float32 arrays (the weight gradients of a layer or
// sub-block that is skipped as a whole).
struct ZeroArgs {
  float* p[6];
  int64_t n[6];
  int32_t count;
};

// Element types of the row kernels: g, y (forward) and gy, gx2 (backward)
// have the configuration's type; the others say theirs (x_f32 etc.), so the
// residual stream and the saved norm inputs can be float32 while the GEMM
// operands are bf16.
struct RmsFwdArgs {
  const void* x;      // source rows (through `src` map)
  RowMap src;
  int32_t x_f32;      // x is float32 (else the configuration's type)
  const void* g;
  float* xcopy;       // optional compacted float32 copy of the source rows
  void* y;            // compacted normalised rows
  float* rstd;        // compacted
  RowCount rc;
  int32_t d;
  float eps;
};

struct RmsBwdArgs {
  const void* x;      // compacted rows
  int32_t x_f32;
  const void* g;
  const float* rstd;
  const void* gy;
  const void* gres;   // optional residual gradient rows (through `res_map`)
  RowMap res_map;
  int32_t gres_f32;
  void* gx;           // output rows through `dst` map
  RowMap dst;
  int32_t gx_f32;
  void* gx2;          // optional second, compacted copy of gx in the configuration's type
  float* dg_part;     // [n_blocks][d]
  RowCount rc;
  int32_t d;
};

struct EltArgs {
  const void* a;
  const void* b;
  void* out;
  RowCount rc;
  int32_t f;
};

struct RowsArgs {
  const void* src;
  void* dst;
  RowMap src_map, dst_map;
  RowCount rc;
  int32_t d;
  float r;
  int32_t src_f32;    // gather: src is float32 (converted to the dtype); else both have the dtype
};

// C[m, n] = (R ? R[m, n] : 0) + alpha * sum_k A(m, k) B(n, k), see ld_gemm.
struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  const void* R;
  int64_t lda, ldb, ldc, ldr;
  int32_t M, N, K;
  const int32_t* dev_count;  // when set: M (count_dim 0) or K (count_dim 1)
  int32_t count_mult;        //   = (*dev_count) * count_mult
  int32_t count_dim;
  RowMap out_map;            // output (and R) row remap; R uses it too when r_mapped
  int32_t r_mapped;
  int32_t r_f32;             // R is float32 (else the configuration's type)
  float alpha;
  const float* alpha_dev;    // when set, alpha is multiplied by *alpha_dev
  int32_t c_f32;
  float* part;               // split-K float32 partials [splits][M][N] (plan.splits > 1)
  // SwiGLU epilogues (256x256 kernels only), d_ff = glu_f:
  //   forward (ld_gemm_bf16_nt_glu_256): B is W_gate_up [2 glu_f, K], N = 2 glu_f;
  //     C receives [u v] rows (ldc = 2 glu_f) and aux the rows of
  //     s = silu(u) v (ld glu_f);
  //   backward (NN part of ld_gemm_bf16_tn_nn_glu_256): N = glu_f; the
  //     product (gs, rounded to bf16) is not stored: aux holds the [u v] rows
  //     (ld 2 glu_f) and C receives [gu gv] rows (ldc = 2 glu_f).
  void* aux;
  int32_t glu_f;
  // Squared-ReLU epilogues (256x256 kernels only) when relu2 is set; aux
  // has leading dimension glu_f (= d_ff):
  //   forward (ld_gemm_bf16_nt_relu2_256): C receives u and aux the rows of
  //     s = relu(u)^2 of the bf16 u;
  //   backward (NN part of ld_gemm_bf16_tn_nn_relu2_256): the product (gs,
  //     rounded to bf16) is not stored: aux holds the u rows and C receives
  //     gu = gs 2 relu(u).
  int32_t relu2;
};

// Kernel choice for one GEMM: the 256x256 MFMA kernel (optionally split
// along K) or the 128x128 one; fp32 uses the SIMT kernel.
struct GemmPlan {
  const char* name;
  int big;
  int splits;
};

struct AttnArgs {
  const void* qkv;
  const void* o;
  const void* go;
  void* out;          // fwd: o ; bwd: gqkv
  float* lse;         // fwd out / bwd in  [n, H, S]
  float* delta;       // bwd: rowsum(dO * O) [n, H, S]
  const int32_t* dev_count;  // kept sequences on the device, or null
  int32_t n_seq;             // host count (upper bound when dev_count is set)
  int32_t S, H, dh;
  float scale;               // 1/sqrt(dh)
  int32_t alibi;             // add the ALiBi bias -m_h (i - j) to the scaled scores
};

// Skinny GEMM of incremental decoding: C[m, n] = (R ? R[m, n] : 0) + alpha *
// sum_k A[m, k] W[n, k], bf16, both operands k-contiguous, M <= kSkinnyMaxM.
struct SkinnyArgs {
  const void* A;
  const void* W;
  void* C;
  const void* R;
  int64_t lda, ldw, ldc, ldr;
  int32_t M, N, K;
  float alpha;
  float* part;        // float32 [ksplit][M][N] when ksplit > 1 or part_only
  int32_t part_only;  // write the partials even with ksplit == 1 (a fused reduction follows)
  // optional: columns kv_d.. of row m also go to the cache kv [*, s_max, 2 kv_d]
  // at position kv_pos + m % kv_n of sequence m / kv_n (the keys/values of a
  // qkv projection)
  void* kv;
  int32_t kv_d, kv_n, kv_s_max, kv_pos;
  // fused decode projection only (launch_gemm_dec): RMSNorm gain applied to
  // the rows of A on load (NULL: A as given), and the activation of the
  // output (kDecAct*; SwiGLU reads gate rows 0..N-1 and up rows N..2N-1 of W)
  const void* g;
  float eps;
  int32_t act;
};
constexpr int kSkinnyMaxM = 64;

// Fused decode projection (at most 8 rows): one workgroup per 8 output
// columns and the whole k range, A rows staged in LDS (normalised on the
// way when g is set); no split-K partials and no separate norm or
// activation launch.
constexpr int kDecGemmMaxM = 8;
constexpr int kDecGemmMaxKNorm = 4096;
constexpr int kDecActNone = 0, kDecActSwiglu = 1, kDecActRelu2 = 2;
// LDS bytes the fused projection needs for K (0 when it does not fit).
size_t dec_gemm_lds_bytes(int64_t K, int nw);
bool dec_gemm_ok(int64_t M, int64_t K, bool norm);
hipError_t launch_gemm_dec(const SkinnyArgs& g, hipStream_t s);

// Copy of the key/value columns of qkv rows into a cache [n_seq, s_max, 2d]
// (keys, then values, of each position): row b*n + j goes to position pos + j
// of sequence b.
struct KvArgs {
  const void* qkv;
  int64_t ld_qkv;
  void* cache;
  int32_t s_max, d, n, n_seq, pos;
};

// Decode attention: queries (rows b*n_new + j of qkv, position pos + j) over
// the cached keys/values of positions 0..pos+n_new-1, in chunks of kDecKeys
// keys with float32 partials combined by a second kernel.
struct DecAttnArgs {
  const void* qkv;
  int64_t ld_qkv;
  const void* cache;
  int32_t s_max;
  void* out;        // [n_seq * n_new, H * dh]
  float* part_o;    // [n_seq][H][n_chunks][kDecMaxRows][dh]
  float* part_ml;   // [n_seq][H][n_chunks][kDecMaxRows][2]: base-2 max, sum
  int32_t n_seq, H, dh, n_new, pos, n_chunks;
  float scale;
  int32_t alibi;
};
constexpr int kDecKeys = 256;
constexpr int kDecMaxRows = 8;

// ALiBi slope of head h of H heads (ALiBi paper, section 3): with n the
// largest power of two <= H, 2^(-8(h+1)/n) for h < n, else every other slope
// of the 2n-head sequence, 2^(-4(2(h-n)+1)/n).
__host__ __device__ inline float alibi_slope(int h, int H) {
  if (H < 1 || h < 0 || h >= H) return 0.f;
  int n = 1;
  while (2 * n <= H) n *= 2;
  const float e = h < n ? -8.f * static_cast<float>(h + 1) / static_cast<float>(n)
                        : -4.f * static_cast<float>(2 * (h - n) + 1) / static_cast<float>(n);
  return exp2f(e);
}

// ------------------------------------------------------------- launchers
// Each returns the HIP error of its launch(es).  Grids are sized for the
// host upper bound; work past the device count exits early.

hipError_t launch_masks(const MaskArgs& a, hipStream_t s);
hipError_t launch_zero_f32(const ZeroArgs& a, hipStream_t s);
int skinny_ksplit(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_skinny(const SkinnyArgs& g, int ksplit, hipStream_t s);
// Fused reductions of a skinny GEMM's partials (g.part_only launches):
// C = bf16(alpha sum + R) and h = RMSNorm(C rows) with gain `gain`; or the
// FFN activation s = act(bf16(alpha sum)) of f columns (SwiGLU pairs
// columns n and f + n).
hipError_t launch_skinny_reduce_norm(const SkinnyArgs& g, int ksplit, const void* gain, float eps, void* h,
                                     hipStream_t s);
hipError_t launch_skinny_reduce_act(const SkinnyArgs& g, int ksplit, int act, int f, void* s_out, hipStream_t s);
hipError_t launch_kv_store(const KvArgs& a, hipStream_t s);
hipError_t launch_attn_decode(const DecAttnArgs& a, hipStream_t s);
hipError_t launch_gather(int dtype, const RowsArgs& a, hipStream_t s);
// n elements between bf16 and float32 (to_f32: bf16 -> float32, else
// float32 -> bf16 with round to nearest even); n % 8 == 0.
hipError_t launch_convert(const void* src, void* dst, int64_t n, int to_f32, hipStream_t s);
hipError_t launch_scatter_add(int dtype, const RowsArgs& a, hipStream_t s);
hipError_t launch_rmsnorm_fwd(int dtype, const RmsFwdArgs& a, hipStream_t s);
// Needs rmsnorm_bwd_blocks(max_rows) * d floats of dg_part.
int64_t rmsnorm_bwd_blocks(int64_t max_rows);
hipError_t launch_rmsnorm_bwd(int dtype, const RmsBwdArgs& a, float* dg, hipStream_t s);
hipError_t launch_relu2_fwd(int dtype, const EltArgs& a, hipStream_t s);
hipError_t launch_relu2_bwd(int dtype, const EltArgs& a, hipStream_t s);
hipError_t launch_swiglu_fwd(int dtype, const EltArgs& a, hipStream_t s);
hipError_t launch_swiglu_bwd(int dtype, const EltArgs& a, hipStream_t s);
hipError_t launch_gemm(int dtype, int a_kcontig, int b_kcontig, const GemmArgs& g, int64_t max_m,
                       int64_t max_k, hipStream_t s);
const char* gemm_kernel_name(int dtype, int a_kcontig, int b_kcontig);
// allow_split: split-K may be chosen (the caller then provides g.part of
// gemm_part_bytes bytes).
GemmPlan plan_gemm(int dtype, int a_kcontig, int b_kcontig, const GemmArgs& g, int64_t max_m,
                   int64_t max_k, bool allow_split);
size_t gemm_part_bytes(const GemmPlan& p, int64_t M, int64_t N);
// Weight-gradient GEMMs g1 and g3 (both operands mn-contiguous, float32
// out; g3 optional and never split, g1 absent when g1.M = 0) and an
// input-gradient GEMM g2 (A k-contiguous, B mn-contiguous) in one launch,
// all of whose plans are the 256x256 kernel.  plan_gemm_pair picks g1's
// split count (at most max_splits) and whether g2's workgroups go first
// from an estimate of the launch's finish time (m3 = 0: no g3); g1.part
// must hold splits1 * M1 * N1 floats when splits1 > 1.
struct PairPlan {
  int splits1;
  int g2_first;
  double est;  // estimated launch time (k-tile times of one CU), reduction included
};
PairPlan plan_gemm_pair(int64_t m1, int64_t n1, int64_t k1, int64_t m3, int64_t n3, int64_t m2, int64_t n2,
                        int64_t k2, int max_splits);
// Launches the kernel only; with p.splits1 > 1 the caller then sums g1's
// partials with launch_splitk_reduce.
hipError_t launch_gemm_pair(GemmArgs g1, const GemmArgs* g3, const PairPlan& p, const GemmArgs& g2, int64_t max_m2,
                            hipStream_t s);
// C[i] = sum over splits of part[s * mn + i] (float32, split order).
hipError_t launch_splitk_reduce(const float* part, int splits, int64_t mn, float* C, hipStream_t s);
// The SwiGLU projection with its activation fused (GemmArgs glu_f, aux):
// ld_gemm_bf16_nt_glu_256 over max_m rows, for bf16 with glu_f % 128 == 0
// and N = 2 glu_f, both operands k-contiguous.
hipError_t launch_gemm_glu_fwd(const GemmArgs& g, int64_t max_m, hipStream_t s);
// ld_gemm_bf16_nt_relu2_256 over max_m rows (see GemmArgs.relu2)
hipError_t launch_gemm_relu2_fwd(const GemmArgs& g, int64_t max_m, hipStream_t s);
hipError_t launch_gemm_plan(int dtype, int a_kcontig, int b_kcontig, const GemmPlan& p, GemmArgs g,
                            int64_t max_m, hipStream_t s);
// Fixed scratch of the no-allocation attention backward (the delta rows,
// one float per (sequence, head, row)), a file-scope device array of this
// many bytes in k_attn.hip.  attn_scratch_ptr gives its address on the
// current device (looked up once per device; no allocation).
constexpr size_t kAttnScratchBytes = size_t(8) << 20;
hipError_t attn_scratch_ptr(float** out);
hipError_t launch_attn_fwd(int dtype, const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_bwd(int dtype, const AttnArgs& a, hipStream_t s);
// The backward kernels one at a time, attn_bwd_parts of them: bf16 0 dQ
// (which also forms delta), 1 dK/dV; float32 0 delta, 1 dK/dV, 2 dQ.
int attn_bwd_parts(int dtype);
hipError_t launch_attn_bwd_part(int dtype, int part, const AttnArgs& a, hipStream_t s);
const char* attn_bwd_kernel_name(int dtype, int part);
const char* attn_fwd_kernel_name(int dtype);

}  // namespace ld

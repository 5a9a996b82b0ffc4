// Host side of the C ABI declared in include/layerdrop.h: argument checks,
// residual scales and integer thresholds, workspace layout, and the order of
// kernel launches for one layer and for a whole training step.  Nothing here
// computes activations or gradients; every step runs in the HIP kernels.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "ld_internal.h"

using namespace ld;

namespace {

// ------------------------------------------------------------------ errors

thread_local std::string t_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return status;
}

#define LD_HIP(call)                                                                    \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) return fail(LD_E_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// --------------------------------------------------------------- profiling

struct ProfRec {
  hipEvent_t e0, e1;
  double flops, bytes;
};

struct Prof {
  std::mutex mu;
  bool on = false;
  std::string name;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  size_t next = 0;
} g_prof;

constexpr size_t kMaxProf = 1 << 16;

bool prof_on() { return g_prof.on; }

// Records events around one launch of kernel `name` when profiling it.
struct ProfScope {
  bool active = false;
  size_t slot = 0;
  hipStream_t s;
  ProfScope(const char* name, hipStream_t st) : s(st) {
    if (!g_prof.on || g_prof.name != name) return;
    if (g_prof.next + 2 > g_prof.pool.size()) {
      if (g_prof.pool.size() >= 2 * kMaxProf) return;
      for (int i = 0; i < 64; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        g_prof.pool.push_back(e);
      }
    }
    slot = g_prof.next;
    g_prof.next += 2;
    active = hipEventRecord(g_prof.pool[slot], s) == hipSuccess;
  }
  void end(double flops, double bytes) {
    if (!active) return;
    if (hipEventRecord(g_prof.pool[slot + 1], s) != hipSuccess) return;
    g_prof.recs.push_back({g_prof.pool[slot], g_prof.pool[slot + 1], flops, bytes});
  }
};

// ------------------------------------------------------------ config checks

struct Dims {
  int64_t B, S, d, H, dh, f, T, es;
  int dtype;
  int kind;    // ld_block_kind
  int64_t fw;  // width of the gate_up GEMM output: 2f (SwiGLU) or f (squared ReLU)
  int sub;     // sub-layer granularity: independent attention / FFN masks
  int per_batch;  // one draw per (layer, step) for the whole batch
  int nm;      // masks per layer: 2 under sub-layer granularity, else 1
};

int check_cfg(const ld_config* c, Dims* out) {
  if (!c) return fail(LD_E_INVALID, "cfg is NULL");
  if (c->batch < 1 || c->seq < 1 || c->d_model < 1 || c->n_heads < 1 || c->d_ff < 1)
    return fail(LD_E_SHAPE, "batch, seq, d_model, n_heads, d_ff must be >= 1");
  if (c->dtype != LD_F32 && c->dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype %d", c->dtype);
  if (c->d_model % c->n_heads) return fail(LD_E_SHAPE, "d_model %% n_heads != 0");
  if (!(c->rms_eps > 0.f) || !std::isfinite(c->rms_eps)) return fail(LD_E_INVALID, "rms_eps must be > 0");
  if (!std::isfinite(c->res_scale)) return fail(LD_E_INVALID, "res_scale must be finite");
  if (c->block_kind != LD_BLOCK_SWIGLU && c->block_kind != LD_BLOCK_ALIBI_RELU2)
    return fail(LD_E_INVALID, "unknown block_kind %d", c->block_kind);
  if (c->granularity < 0 || c->granularity > 3)
    return fail(LD_E_INVALID, "unknown granularity %d", c->granularity);
  const int dh = c->d_model / c->n_heads;
  if (c->dtype == LD_BF16) {
    if (dh != 64 && dh != 128) return fail(LD_E_UNSUPPORTED, "bf16 needs d_head 64 or 128, got %d", dh);
    if (c->d_model % 8 || c->d_ff % 8) return fail(LD_E_SHAPE, "bf16 needs d_model, d_ff multiples of 8");
    if (c->seq % 64) return fail(LD_E_SHAPE, "bf16 needs seq %% 64 == 0");
    if (c->d_model > 4096) return fail(LD_E_UNSUPPORTED, "d_model > 4096");
  } else {
    if (dh != 16 && dh != 32 && dh != 64)
      return fail(LD_E_UNSUPPORTED, "fp32 needs d_head 16, 32 or 64, got %d", dh);
    if (c->d_model % 4 || c->d_ff % 4) return fail(LD_E_SHAPE, "fp32 needs d_model, d_ff multiples of 4");
    if (c->d_model > 2048) return fail(LD_E_UNSUPPORTED, "d_model > 2048");
  }
  const int64_t T = static_cast<int64_t>(c->batch) * c->seq;
  if (T * std::max<int64_t>(3ll * c->d_model, 2ll * c->d_ff) >= (1ll << 40) || T >= (1ll << 30))
    return fail(LD_E_SHAPE, "batch * seq too large");
  if (out) {
    out->B = c->batch;
    out->S = c->seq;
    out->d = c->d_model;
    out->H = c->n_heads;
    out->dh = dh;
    out->f = c->d_ff;
    out->T = T;
    out->es = c->dtype == LD_BF16 ? 2 : 4;
    out->dtype = c->dtype;
    out->kind = c->block_kind;
    out->fw = c->block_kind == LD_BLOCK_SWIGLU ? 2ll * c->d_ff : c->d_ff;
    out->sub = c->granularity & LD_GRAN_SUBLAYER ? 1 : 0;
    out->per_batch = c->granularity & LD_GRAN_PER_BATCH ? 1 : 0;
    out->nm = out->sub ? 2 : 1;
  }
  return LD_OK;
}

int check_p(float p) {
  if (std::isnan(p) || p < 0.f || p > 1.f) return fail(LD_E_INVALID, "p = %g outside [0, 1]", p);
  return LD_OK;
}

// Integer drop threshold: drop iff word < thr; p >= 1 drops all.
void threshold(float p, uint64_t* thr, uint8_t* drop_all) {
  *drop_all = 0;
  *thr = 0;
  if (p >= 1.f) {
    *drop_all = 1;
    return;
  }
  if (p <= 0.f) return;
  *thr = static_cast<uint64_t>(std::floor(std::ldexp(static_cast<double>(p), 64)));
}

// r for a layer; 0 when nothing can be kept (it is then never applied).
float residual_scale(const ld_config* c, float p) {
  if (p >= 1.f) return 0.f;
  if (!c->rescale) return c->res_scale;
  return static_cast<float>(static_cast<double>(c->res_scale) / (1.0 - static_cast<double>(p)));
}

// ------------------------------------------------------------------ layout

constexpr size_t kAlign = 256;
size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Saved activations of one layer, sized for the whole batch (kept rows are
// stored compacted from row 0).  xk (the layer input rows) and zk (Z, the
// input of the FFN sub-block) are float32 in every configuration: they are
// the residual stream inside the layer and the norm inputs of the backward.
struct ActLayout {
  size_t xk, rstd1, h1, qkv, att, lse, zk, rstd2, h2, uv, s, total;
};

ActLayout act_layout(const Dims& D) {
  ActLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += up(bytes);
    return at;
  };
  const size_t es = D.es, T = D.T;
  L.xk = take(4 * T * D.d);
  L.rstd1 = take(4 * T);
  L.h1 = take(es * T * D.d);
  L.qkv = take(es * T * 3 * D.d);
  L.att = take(es * T * D.d);
  L.lse = take(4 * T * D.H);
  L.zk = take(4 * T * D.d);
  L.rstd2 = take(4 * T);
  L.h2 = take(es * T * D.d);
  L.uv = take(es * T * D.fw);
  L.s = take(es * T * D.f);
  L.total = o;
  return L;
}

// Mask block of one layer inside a ld_layer_fwd ctx.
struct MaskLayout {
  size_t keep, idx, count, r, total;
};

// nm masks per layer (attention, FFN under sub-layer granularity), stored
// [layer][mask][batch].
MaskLayout mask_layout(int64_t L, int64_t B, int64_t nm) {
  MaskLayout m{};
  size_t o = 0;
  m.keep = o;
  o += up(L * nm * B);
  m.idx = o;
  o += up(4 * L * nm * B);
  m.count = o;
  o += up(4 * L * nm);
  m.r = o;
  o += up(4 * L);
  m.total = o;
  return m;
}

// Split-K float32 scratch for the weight-gradient GEMMs (largest of the four).
size_t splitk_bytes(const Dims& D) {
  if (D.dtype != LD_BF16) return 0;
  const int64_t shapes[4][2] = {{D.d, D.f}, {D.fw, D.d}, {D.d, D.d}, {3 * D.d, D.d}};
  size_t best = 0;
  for (const auto& sh : shapes) {
    GemmArgs g;
    std::memset(&g, 0, sizeof(g));
    g.M = static_cast<int32_t>(sh[0]);
    g.N = static_cast<int32_t>(sh[1]);
    g.ldc = g.N;
    g.c_f32 = 1;
    const GemmPlan p = plan_gemm(D.dtype, 0, 0, g, sh[0], D.T, true);
    best = std::max(best, gemm_part_bytes(p, sh[0], sh[1]));
  }
  return best;
}

// Backward scratch.  gz32: dL/dZ of the kept rows in float32 (the residual
// gradient inside the layer); gz: the same rows in the configuration's type
// (the operand of the output projection's backward GEMMs; unused in float32
// configurations, where gz32 serves both).
struct BwdLayout {
  size_t gk, gs, guv, gh, gz, gz32, ga, gqkv, delta, dg_part, splitk, splitk_bytes, total;
};

BwdLayout bwd_layout(const Dims& D) {
  BwdLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += up(bytes);
    return at;
  };
  const size_t es = D.es, T = D.T;
  L.gk = take(es * T * D.d);
  L.gs = take(es * T * D.f);
  L.guv = take(es * T * D.fw);
  L.gh = take(es * T * D.d);
  L.gz = take(es * T * D.d);
  L.gz32 = take(4 * T * D.d);
  L.ga = take(es * T * D.d);
  L.gqkv = take(es * T * 3 * D.d);
  L.delta = take(4 * T * D.H);
  L.dg_part = take(4 * rmsnorm_bwd_blocks(T) * D.d);
  L.splitk_bytes = splitk_bytes(D);
  L.splitk = take(L.splitk_bytes);
  L.total = o;
  return L;
}

// Pointers of one sub-block's mask data on the device.  With count null
// every row is processed (evaluation form: no masks), idx null is the
// identity map, and r null means the host scale r_host.
struct MaskView {
  const uint8_t* keep;
  const int32_t* idx;
  const int32_t* count;
  const float* r;
  float r_host = 1.f;
};

// The masks of one layer: attention and FFN views (the same view under layer
// granularity), what the host knows of them (-1: decided on the device;
// 0: dropped for the whole batch; 1: kept for the whole batch, from the
// per-batch draw), and the kept counts while profiling (-1 otherwise).
struct LayerMasks {
  MaskView a, f;
  int host_a, host_f;
  int64_t hc_a, hc_f;
};

// A residual stream: x (forward) or dL/dx (backward) rows [B, S, d], float32
// or the configuration's type.  ld_layer_fwd / ld_layer_bwd run on the
// caller's tensors; ld_stack_step on float32 copies of them in its
// workspace, so the stream is rounded to the caller's type only once.
struct Stream {
  void* p;
  int f32;
};

struct ActPtrs {
  char* base;
  ActLayout L;
  template <typename T = void>
  T* at(size_t off) const {
    return reinterpret_cast<T*>(base + off);
  }
};

// Kept counts on the host, read back only while profiling (one stream sync).
std::vector<int64_t> host_counts_if_profiling(const int32_t* dev_count, int64_t n, hipStream_t s) {
  std::vector<int64_t> out(n, -1);
  if (!prof_on()) return out;
  std::vector<int32_t> c(n, 0);
  if (hipMemcpyAsync(c.data(), dev_count, sizeof(int32_t) * n, hipMemcpyDeviceToHost, s) != hipSuccess)
    return out;
  if (hipStreamSynchronize(s) != hipSuccess) return out;
  for (int64_t i = 0; i < n; ++i) out[i] = c[i];
  return out;
}

// ----------------------------------------------------------- gemm helper

struct GemmCall {
  int dtype;
  int a_k, b_k;
  GemmArgs g;
  int64_t max_m;
};

GemmArgs gemm_args() {
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.alpha = 1.f;
  return g;
}

// part: split-K scratch of part_bytes bytes (may be null / 0: no split).
int run_gemm(int dtype, int a_k, int b_k, GemmArgs g, int64_t max_m, int64_t host_m,
             int64_t host_k, hipStream_t s, float* part = nullptr, size_t part_bytes = 0,
             int64_t max_k = 0) {
  const GemmPlan plan = plan_gemm(dtype, a_k, b_k, g, max_m, max_k, part != nullptr);
  if (plan.splits > 1) {
    if (gemm_part_bytes(plan, g.M, g.N) > part_bytes) return fail(LD_E_WORKSPACE, "split-K scratch too small");
    g.part = part;
  }
  const char* name = plan.name;
  ProfScope ps(name, s);
  hipError_t e = launch_gemm_plan(dtype, a_k, b_k, plan, g, max_m, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "%s launch: %s", name, hipGetErrorString(e));
  const double es = dtype == LD_BF16 ? 2.0 : 4.0;
  const double M = static_cast<double>(host_m), N = g.N, K = static_cast<double>(host_k);
  const double out_es = g.c_f32 ? 4.0 : es;
  const double r_es = g.r_f32 ? 4.0 : es;
  ps.end(2.0 * M * N * K, es * (M * K + N * K) + out_es * M * N + (g.R ? r_es * M * N : 0.0));
  return LD_OK;
}

// Weight-gradient GEMMs (g1, and g3 when given: both operands mn-contiguous,
// float32 out, their reduction length the kept rows) and an input-gradient
// GEMM (g2: A k-contiguous, B mn-contiguous) in one launch when all take the
// 256x256 kernel; otherwise one after the other.  g1.M = 0: no g1.
bool gemm_pair_ok(int dtype, const GemmArgs& g1, int64_t max_k1, const GemmArgs& g2, int64_t max_m2,
                  const GemmArgs* g3 = nullptr) {
  return dtype == LD_BF16 && (g1.M == 0 || plan_gemm(dtype, 0, 0, g1, g1.M, max_k1, true).big) &&
         (!g3 || plan_gemm(dtype, 0, 0, *g3, g3->M, max_k1, false).big) &&
         plan_gemm(dtype, 1, 0, g2, max_m2, 0, false).big;
}

// The plan run_gemm_pair takes for these GEMMs (the 256x256 kernels).
PairPlan pair_plan(int dtype, const GemmArgs& g1, int64_t host_k1, int64_t max_k1, const GemmArgs& g2,
                   int64_t max_m2, int64_t host_m2, bool can_split, const GemmArgs* g3 = nullptr) {
  const bool has1 = g1.M > 0;
  const int max_splits = has1 ? plan_gemm(dtype, 0, 0, g1, g1.M, max_k1, can_split).splits : 1;
  const int64_t plan_k1 = host_k1 >= 0 ? host_k1 : max_k1, plan_m2 = host_m2 >= 0 ? host_m2 : max_m2;
  return plan_gemm_pair(has1 ? g1.M : 0, g1.N, plan_k1, g3 ? g3->M : 0, g3 ? g3->N : 0, plan_m2, g2.N, g2.K,
                        max_splits);
}

// Whether the backward of a sub-block runs its input-gradient GEMM gA alone
// and puts its weight gradient wA into the launch of (wB, gB) -- three
// GEMMs in one launch -- rather than the two pairs (wA, gA) and (wB, gB):
// when all take the 256x256 kernels and the launches' estimated times say
// so for these kept rows.
bool group_weight_grads(int dtype, const GemmArgs& wA, const GemmArgs& gA, const GemmArgs& wB, const GemmArgs& gB,
                        int64_t host_k, int64_t T, bool can_split) {
  const GemmArgs none = gemm_args();
  if (host_k < 0 || !gemm_pair_ok(dtype, wA, T, gA, T) || !gemm_pair_ok(dtype, none, T, gA, T) ||
      !gemm_pair_ok(dtype, wB, T, gB, T, &wA))
    return false;
  const double pairs = pair_plan(dtype, wA, host_k, T, gA, T, host_k, can_split).est +
                       pair_plan(dtype, wB, host_k, T, gB, T, host_k, can_split).est;
  const double grouped = pair_plan(dtype, none, host_k, T, gA, T, host_k, can_split).est +
                         pair_plan(dtype, wB, host_k, T, gB, T, host_k, can_split, &wA).est;
  return grouped < pairs;
}

// g2.glu_f > 0 (only when gemm_pair_ok): the SwiGLU backward is fused into
// g2's epilogue (see GemmArgs).
int run_gemm_pair(int dtype, GemmArgs g1, int64_t host_k1, int64_t max_k1, GemmArgs g2, int64_t max_m2,
                  int64_t host_m2, int64_t host_k2, hipStream_t s, float* part, size_t part_bytes,
                  const GemmArgs* g3 = nullptr) {
  const bool has1 = g1.M > 0;
  if (!gemm_pair_ok(dtype, g1, max_k1, g2, max_m2, g3)) {
    if (g2.glu_f > 0 || g2.relu2) return fail(LD_E_INVALID, "a fused activation backward needs the paired 256x256 kernels");
    if (int rc = run_gemm(dtype, 1, 0, g2, max_m2, host_m2, host_k2, s)) return rc;
    if (has1)
      if (int rc = run_gemm(dtype, 0, 0, g1, g1.M, g1.M, host_k1, s, part, part_bytes, max_k1)) return rc;
    if (g3) return run_gemm(dtype, 0, 0, *g3, g3->M, g3->M, host_k1, s, part, part_bytes, max_k1);
    return LD_OK;
  }
  // at most the split count the standalone plan (and the scratch) allows,
  // planned for the kept rows when the host knows them (the grid still
  // covers max_m2 rows; the device counts decide which work)
  const PairPlan pp = pair_plan(dtype, g1, host_k1, max_k1, g2, max_m2, host_m2, part != nullptr, g3);
  if (pp.splits1 > 1) {
    GemmPlan q = plan_gemm(dtype, 0, 0, g1, g1.M, max_k1, true);
    q.splits = pp.splits1;
    if (gemm_part_bytes(q, g1.M, g1.N) > part_bytes) return fail(LD_E_WORKSPACE, "split-K scratch too small");
    g1.part = part;
  }
  const char* name = g2.relu2 ? "ld_gemm_bf16_tn_nn_relu2_256"
                    : g2.glu_f > 0 ? "ld_gemm_bf16_tn_nn_glu_256" : "ld_gemm_bf16_tn_nn_256";
  ProfScope ps(name, s);
  const hipError_t e = launch_gemm_pair(g1, g3, pp, g2, max_m2, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "%s launch: %s", name, hipGetErrorString(e));
  const double K1 = static_cast<double>(host_k1);
  const double M2 = static_cast<double>(host_m2), N2 = g2.N, K2 = static_cast<double>(host_k2);
  const double mn1 = has1 ? static_cast<double>(g1.M) * g1.N : 0.0, mn3 = g3 ? static_cast<double>(g3->M) * g3->N : 0.0;
  const double mk1 = has1 ? static_cast<double>(g1.M + g1.N) : 0.0, mk3 = g3 ? static_cast<double>(g3->M + g3->N) : 0.0;
  // a fused epilogue reads [u v] and writes [gu gv] (u and gu with squared
  // ReLU) instead of writing gs
  const double out2 = g2.relu2 ? 2.0 * M2 * N2 : g2.glu_f > 0 ? 4.0 * M2 * N2 : 1.0 * M2 * N2;
  ps.end(2.0 * ((mn1 + mn3) * K1 + M2 * N2 * K2),
         2.0 * (mk1 + mk3) * K1 + 4.0 * (mn1 * pp.splits1 + mn3) + 2.0 * (M2 * K2 + N2 * K2 + out2));
  if (pp.splits1 > 1) {
    const int64_t mn = static_cast<int64_t>(g1.M) * g1.N;
    ProfScope pr("ld_splitk_reduce", s);
    const hipError_t er = launch_splitk_reduce(g1.part, pp.splits1, mn, static_cast<float*>(g1.C), s);
    if (er != hipSuccess) return fail(LD_E_HIP, "ld_splitk_reduce launch: %s", hipGetErrorString(er));
    pr.end(0, 4.0 * mn * (pp.splits1 + 1.0));
  }
  return LD_OK;
}

// ------------------------------------------------------------ one layer

// Attention sub-block on the rows mv keeps.  hc: its kept count when
// profiling (read back by the caller), else -1.  scatter = 0 leaves
// Z = X + r f_attn(X) compacted in act (zk) for the FFN sub-block of the same
// rows; scatter = 1 writes Z into the kept rows of x (sub-layer granularity,
// where the FFN keeps its own rows).
// kv: null, or a cache [B, s_max, 2d] that receives the keys and values of
// positions 0..S-1 (evaluation form only: every sequence processed).
int attn_forward_part(const ld_config* cfg, const Dims& D, const ld_weights& w, const MaskView& mv,
                      const ActPtrs& act, Stream xs, int64_t hc, bool scatter, hipStream_t s,
                      void* kv = nullptr, int32_t s_max = 0) {
  const int dt = D.dtype;
  const int64_t T = D.T;
  const int64_t hm = hc * D.S;
  hipError_t e;

  // gather kept rows of X + RMSNorm (attention input)
  {
    RmsFwdArgs a{};
    a.x = xs.p;
    a.x_f32 = xs.f32;
    a.src = {mv.idx, static_cast<int32_t>(D.S)};
    a.g = w.g_attn;
    a.xcopy = act.at<float>(act.L.xk);
    a.y = act.at(act.L.h1);
    a.rstd = act.at<float>(act.L.rstd1);
    a.rc = {mv.count, static_cast<int32_t>(D.S), T};
    a.d = static_cast<int32_t>(D.d);
    a.eps = cfg->rms_eps;
    ProfScope ps("ld_rmsnorm_fwd_k", s);
    if ((e = launch_rmsnorm_fwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "rmsnorm_fwd: %s", hipGetErrorString(e));
    ps.end(0, (xs.f32 ? 4.0 : D.es) * hm * D.d + 4.0 * hm * D.d + D.es * hm * D.d + 4.0 * hm);
  }
  // qkv = h1 W_qkv^T
  {
    GemmArgs g = gemm_args();
    g.A = act.at(act.L.h1);
    g.lda = D.d;
    g.B = w.w_qkv;
    g.ldb = D.d;
    g.C = act.at(act.L.qkv);
    g.ldc = 3 * D.d;
    g.N = static_cast<int32_t>(3 * D.d);
    g.K = static_cast<int32_t>(D.d);
    g.M = static_cast<int32_t>(T);
    g.dev_count = mv.count;
    g.count_mult = static_cast<int32_t>(D.S);
    if (int rc = run_gemm(dt, 1, 1, g, T, hm, D.d, s)) return rc;
  }
  if (kv) {
    KvArgs k{};
    k.qkv = act.at(act.L.qkv);
    k.ld_qkv = 3 * D.d;
    k.cache = kv;
    k.s_max = s_max;
    k.d = static_cast<int32_t>(D.d);
    k.n = static_cast<int32_t>(D.S);
    k.n_seq = static_cast<int32_t>(D.B);
    k.pos = 0;
    ProfScope ps("ld_kv_store_k", s);
    if ((e = launch_kv_store(k, s)) != hipSuccess) return fail(LD_E_HIP, "kv store: %s", hipGetErrorString(e));
    ps.end(0, 2.0 * D.es * hm * 2 * D.d);
  }
  // causal attention on the kept sequences
  {
    AttnArgs a{};
    a.qkv = act.at(act.L.qkv);
    a.out = act.at(act.L.att);
    a.lse = act.at<float>(act.L.lse);
    a.dev_count = mv.count;
    a.n_seq = static_cast<int32_t>(D.B);
    a.S = static_cast<int32_t>(D.S);
    a.H = static_cast<int32_t>(D.H);
    a.dh = static_cast<int32_t>(D.dh);
    a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(D.dh)));
    a.alibi = D.kind == LD_BLOCK_ALIBI_RELU2;
    ProfScope ps(attn_fwd_kernel_name(dt), s);
    if ((e = launch_attn_fwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "attn_fwd: %s", hipGetErrorString(e));
    ps.end(2.0 * hc * D.d * D.S * (D.S + 1.0), D.es * hm * D.d * 4.0);
  }
  // zk = xk + r * (att W_o^T) (float32), or x[kept rows] = the same
  {
    GemmArgs g = gemm_args();
    g.A = act.at(act.L.att);
    g.lda = D.d;
    g.B = w.w_o;
    g.ldb = D.d;
    g.C = scatter ? xs.p : act.at(act.L.zk);
    g.c_f32 = scatter ? xs.f32 : 1;
    g.ldc = D.d;
    g.R = act.at(act.L.xk);
    g.r_f32 = 1;
    g.ldr = D.d;
    if (scatter) {
      g.r_mapped = 0;
      g.out_map = {mv.idx, static_cast<int32_t>(D.S)};
    }
    g.alpha_dev = mv.r;
    if (!mv.r) g.alpha = mv.r_host;
    g.N = static_cast<int32_t>(D.d);
    g.K = static_cast<int32_t>(D.d);
    g.M = static_cast<int32_t>(T);
    g.dev_count = mv.count;
    g.count_mult = static_cast<int32_t>(D.S);
    if (int rc = run_gemm(dt, 1, 1, g, T, hm, D.d, s)) return rc;
  }
  return LD_OK;
}

// FFN sub-block on the rows mv keeps, written into x.  gather = 0 reads Z from
// act (zk, left there by attn_forward_part for the same rows); gather = 1
// reads the kept rows of x (which then holds Z) and saves them to zk.
int ffn_forward_part(const ld_config* cfg, const Dims& D, const ld_weights& w, const MaskView& mv,
                     const ActPtrs& act, Stream xs, int64_t hc, bool gather, hipStream_t s) {
  const int dt = D.dtype;
  const int64_t T = D.T;
  const int64_t hm = hc * D.S;
  hipError_t e;
  // RMSNorm (FFN input)
  {
    RmsFwdArgs a{};
    if (gather) {
      a.x = xs.p;
      a.x_f32 = xs.f32;
      a.src = {mv.idx, static_cast<int32_t>(D.S)};
      a.xcopy = act.at<float>(act.L.zk);
    } else {
      a.x = act.at(act.L.zk);
      a.x_f32 = 1;
      a.src = {nullptr, 1};
    }
    a.g = w.g_mlp;
    a.y = act.at(act.L.h2);
    a.rstd = act.at<float>(act.L.rstd2);
    a.rc = {mv.count, static_cast<int32_t>(D.S), T};
    a.d = static_cast<int32_t>(D.d);
    a.eps = cfg->rms_eps;
    ProfScope ps("ld_rmsnorm_fwd_k", s);
    if ((e = launch_rmsnorm_fwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "rmsnorm_fwd: %s", hipGetErrorString(e));
    ps.end(0, (gather ? (xs.f32 ? 4.0 : D.es) + 4.0 : 4.0) * hm * D.d + D.es * hm * D.d + 4.0 * hm);
  }
  // [u v] = h2 W_gate_up^T (SwiGLU), u = h2 W_up^T (squared ReLU)
  {
    GemmArgs g = gemm_args();
    g.A = act.at(act.L.h2);
    g.lda = D.d;
    g.B = w.w_gate_up;
    g.ldb = D.d;
    g.C = act.at(act.L.uv);
    g.ldc = D.fw;
    g.N = static_cast<int32_t>(D.fw);
    g.K = static_cast<int32_t>(D.d);
    g.M = static_cast<int32_t>(T);
    g.dev_count = mv.count;
    g.count_mult = static_cast<int32_t>(D.S);
    // SwiGLU fused into the projection's epilogue where the 256x256 kernel
    // applies and d_ff is a multiple of 128
    if (D.kind == LD_BLOCK_SWIGLU && dt == LD_BF16 && D.f % 128 == 0 && plan_gemm(dt, 1, 1, g, T, 0, false).big) {
      g.aux = act.at(act.L.s);
      g.glu_f = static_cast<int32_t>(D.f);
      ProfScope ps("ld_gemm_bf16_nt_glu_256", s);
      if ((e = launch_gemm_glu_fwd(g, T, s)) != hipSuccess)
        return fail(LD_E_HIP, "ld_gemm_bf16_nt_glu_256 launch: %s", hipGetErrorString(e));
      ps.end(2.0 * hm * D.fw * D.d, D.es * (hm * D.d + D.fw * D.d + hm * D.fw + hm * D.f));
      goto down_projection;
    }
    // squared ReLU likewise (u and s from one epilogue)
    if (D.kind == LD_BLOCK_ALIBI_RELU2 && dt == LD_BF16 && plan_gemm(dt, 1, 1, g, T, 0, false).big) {
      g.aux = act.at(act.L.s);
      g.glu_f = static_cast<int32_t>(D.f);
      g.relu2 = 1;
      ProfScope ps("ld_gemm_bf16_nt_relu2_256", s);
      if ((e = launch_gemm_relu2_fwd(g, T, s)) != hipSuccess)
        return fail(LD_E_HIP, "ld_gemm_bf16_nt_relu2_256 launch: %s", hipGetErrorString(e));
      ps.end(2.0 * hm * D.fw * D.d, D.es * (hm * D.d + D.fw * D.d + 2.0 * hm * D.f));
      goto down_projection;
    }
    if (int rc = run_gemm(dt, 1, 1, g, T, hm, D.d, s)) return rc;
  }
  // s = silu(u) * v  or  s = relu(u)^2
  {
    EltArgs a{};
    a.a = act.at(act.L.uv);
    a.out = act.at(act.L.s);
    a.rc = {mv.count, static_cast<int32_t>(D.S), T};
    a.f = static_cast<int32_t>(D.f);
    if (D.kind == LD_BLOCK_SWIGLU) {
      ProfScope ps("ld_swiglu_fwd_k", s);
      if ((e = launch_swiglu_fwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "swiglu_fwd: %s", hipGetErrorString(e));
      ps.end(0, D.es * hm * D.f * 3.0);
    } else {
      ProfScope ps("ld_relu2_fwd_k", s);
      if ((e = launch_relu2_fwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "relu2_fwd: %s", hipGetErrorString(e));
      ps.end(0, D.es * hm * D.f * 2.0);
    }
  }
down_projection:
  // X[kept rows] = zk + r * (s W_down^T)  (scatter into the residual stream)
  {
    GemmArgs g = gemm_args();
    g.A = act.at(act.L.s);
    g.lda = D.f;
    g.B = w.w_down;
    g.ldb = D.f;
    g.C = xs.p;
    g.c_f32 = xs.f32;
    g.ldc = D.d;
    g.R = act.at(act.L.zk);
    g.r_f32 = 1;
    g.ldr = D.d;
    g.r_mapped = 0;
    g.out_map = {mv.idx, static_cast<int32_t>(D.S)};
    g.alpha_dev = mv.r;
    if (!mv.r) g.alpha = mv.r_host;
    g.N = static_cast<int32_t>(D.d);
    g.K = static_cast<int32_t>(D.f);
    g.M = static_cast<int32_t>(T);
    g.dev_count = mv.count;
    g.count_mult = static_cast<int32_t>(D.S);
    if (int rc = run_gemm(dt, 1, 1, g, T, hm, D.f, s)) return rc;
  }
  return LD_OK;
}

// Weight gradients of a sub-block skipped for the whole batch: zeros.
int zero_grads(const Dims& D, const ld_grads& dw, bool attn, bool ffn, hipStream_t s) {
  ZeroArgs z{};
  if (attn) {
    z.p[z.count] = dw.g_attn, z.n[z.count++] = D.d;
    z.p[z.count] = dw.w_qkv, z.n[z.count++] = 3 * D.d * D.d;
    z.p[z.count] = dw.w_o, z.n[z.count++] = D.d * D.d;
  }
  if (ffn) {
    z.p[z.count] = dw.g_mlp, z.n[z.count++] = D.d;
    z.p[z.count] = dw.w_gate_up, z.n[z.count++] = D.fw * D.d;
    z.p[z.count] = dw.w_down, z.n[z.count++] = D.d * D.f;
  }
  if (!z.count) return LD_OK;
  ProfScope ps("ld_zero_f32_k", s);
  hipError_t e = launch_zero_f32(z, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "zero fill: %s", hipGetErrorString(e));
  double n = 0;
  for (int i = 0; i < z.count; ++i) n += static_cast<double>(z.n[i]);
  ps.end(0, 4.0 * n);
  return LD_OK;
}

// One layer forward.  Layer granularity: both sub-blocks on the same rows, Z
// kept compacted between them.  Sub-layer granularity: each sub-block on its
// own rows, Z passed through x.  A sub-block the host knows to be dropped for
// the whole batch launches nothing.
int layer_forward(const ld_config* cfg, const Dims& D, const ld_weights& w, const LayerMasks& lm,
                  const ActPtrs& act, Stream xs, hipStream_t s) {
  if (!D.sub) {
    if (lm.host_a == 0) return LD_OK;
    if (int rc = attn_forward_part(cfg, D, w, lm.a, act, xs, lm.hc_a, false, s)) return rc;
    return ffn_forward_part(cfg, D, w, lm.a, act, xs, lm.hc_a, false, s);
  }
  if (lm.host_a != 0)
    if (int rc = attn_forward_part(cfg, D, w, lm.a, act, xs, lm.hc_a, true, s)) return rc;
  if (lm.host_f != 0)
    if (int rc = ffn_forward_part(cfg, D, w, lm.f, act, xs, lm.hc_f, true, s)) return rc;
  return LD_OK;
}

// Backward of ffn_forward_part on the rows mv keeps, given dL/dX^{l+1} in
// the gradient stream ds.  scatter = 0 leaves dL/dZ of those rows compacted
// in the scratch (gz32, and gz in bf16) for the attention sub-block of the
// same rows; scatter = 1 writes it into the kept rows of the stream
// (sub-layer granularity).
int ffn_backward_part(const Dims& D, const ld_weights& w, const MaskView& mv, const ActPtrs& act,
                      const BwdLayout& BL, char* ws, Stream ds, const ld_grads& dw, int64_t hc,
                      bool scatter, hipStream_t s) {
  const int dt = D.dtype;
  const int64_t T = D.T;
  const int64_t hm = hc * D.S;
  const int32_t S = static_cast<int32_t>(D.S);
  auto W = [&](size_t off) { return static_cast<void*>(ws + off); };
  float* SK = BL.splitk_bytes ? reinterpret_cast<float*>(ws + BL.splitk) : nullptr;
  hipError_t e;

  // gk = dL/dX^{l+1} on the kept rows, in the configuration's type (the
  // operand of the down projection's backward GEMMs)
  {
    RowsArgs a{};
    a.src = ds.p;
    a.src_f32 = ds.f32;
    a.dst = W(BL.gk);
    a.src_map = {mv.idx, S};
    a.dst_map = {nullptr, 1};
    a.rc = {mv.count, S, T};
    a.d = static_cast<int32_t>(D.d);
    ProfScope ps("ld_gather_rows_k", s);
    if ((e = launch_gather(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "gather: %s", hipGetErrorString(e));
    ps.end(0, ((ds.f32 ? 4.0 : D.es) + D.es) * hm * D.d);
  }
  // gs = r * gk W_down [M, f] and dW_down = r * gk^T s [d, f]; gh2 = guv
  // W_gate_up [M, d] and dW_gate_up = guv^T h2 [fw, d].  With the 256x256
  // kernels the activation's backward is fused into gs's epilogue (guv from
  // gs without storing gs), and dW_down waits for the gate/up launch, which
  // then holds both weight gradients (mostly without split-K).
  GemmArgs g_gs = gemm_args();
  g_gs.A = W(BL.gk);
  g_gs.lda = D.d;
  g_gs.B = w.w_down;
  g_gs.ldb = D.f;
  g_gs.C = W(BL.gs);
  g_gs.ldc = D.f;
  g_gs.alpha_dev = mv.r;
  g_gs.N = static_cast<int32_t>(D.f);
  g_gs.K = static_cast<int32_t>(D.d);
  g_gs.dev_count = mv.count;
  g_gs.count_mult = S;
  GemmArgs g_wd = gemm_args();
  g_wd.A = W(BL.gk);
  g_wd.lda = D.d;
  g_wd.B = act.at(act.L.s);
  g_wd.ldb = D.f;
  g_wd.C = dw.w_down;
  g_wd.ldc = D.f;
  g_wd.c_f32 = 1;
  g_wd.alpha_dev = mv.r;
  g_wd.M = static_cast<int32_t>(D.d);
  g_wd.N = static_cast<int32_t>(D.f);
  g_wd.dev_count = mv.count;
  g_wd.count_mult = S;
  g_wd.count_dim = 1;
  GemmArgs g_gh2 = gemm_args();
  g_gh2.A = W(BL.guv);
  g_gh2.lda = D.fw;
  g_gh2.B = w.w_gate_up;
  g_gh2.ldb = D.d;
  g_gh2.C = W(BL.gh);
  g_gh2.ldc = D.d;
  g_gh2.N = static_cast<int32_t>(D.d);
  g_gh2.K = static_cast<int32_t>(D.fw);
  g_gh2.dev_count = mv.count;
  g_gh2.count_mult = S;
  GemmArgs g_wgu = gemm_args();
  g_wgu.A = W(BL.guv);
  g_wgu.lda = D.fw;
  g_wgu.B = act.at(act.L.h2);
  g_wgu.ldb = D.d;
  g_wgu.C = dw.w_gate_up;
  g_wgu.ldc = D.d;
  g_wgu.c_f32 = 1;
  g_wgu.M = static_cast<int32_t>(D.fw);
  g_wgu.N = static_cast<int32_t>(D.d);
  g_wgu.dev_count = mv.count;
  g_wgu.count_mult = S;
  g_wgu.count_dim = 1;
  const GemmArgs none = gemm_args();  // M = 0: no weight gradient in the launch
  const bool act_fused = gemm_pair_ok(dt, g_wd, T, g_gs, T);
  const bool grouped = act_fused && group_weight_grads(dt, g_wd, g_gs, g_wgu, g_gh2, hm, T, SK != nullptr);
  if (act_fused) {
    g_gs.C = W(BL.guv);
    g_gs.ldc = D.fw;
    g_gs.aux = act.at(act.L.uv);
    g_gs.glu_f = static_cast<int32_t>(D.f);
    g_gs.relu2 = D.kind == LD_BLOCK_ALIBI_RELU2;
  }
  if (int rc = run_gemm_pair(dt, grouped ? none : g_wd, hm, T, g_gs, T, hm, D.d, s, SK, BL.splitk_bytes)) return rc;
  // guv = SwiGLU backward, or gu = squared-ReLU backward
  if (!act_fused) {
    EltArgs a{};
    a.a = act.at(act.L.uv);
    a.b = W(BL.gs);
    a.out = W(BL.guv);
    a.rc = {mv.count, S, T};
    a.f = static_cast<int32_t>(D.f);
    if (D.kind == LD_BLOCK_SWIGLU) {
      ProfScope ps("ld_swiglu_bwd_k", s);
      if ((e = launch_swiglu_bwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "swiglu_bwd: %s", hipGetErrorString(e));
      ps.end(0, D.es * hm * D.f * 5.0);
    } else {
      ProfScope ps("ld_relu2_bwd_k", s);
      if ((e = launch_relu2_bwd(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "relu2_bwd: %s", hipGetErrorString(e));
      ps.end(0, D.es * hm * D.f * 3.0);
    }
  }
  if (int rc = run_gemm_pair(dt, g_wgu, hm, T, g_gh2, T, hm, D.fw, s, SK, BL.splitk_bytes, grouped ? &g_wd : nullptr))
    return rc;
  // gz = dL/dX^{l+1} + RMSNorm_bwd(zk, g_mlp, gh2); dg_mlp.  The residual
  // gradient is read from the stream itself; gz goes to gz32 (float32) and,
  // in bf16 configurations, to gz (the operand of the next GEMMs) -- or,
  // under sub-layer granularity, back into the stream.
  {
    RmsBwdArgs a{};
    a.x = act.at(act.L.zk);
    a.x_f32 = 1;
    a.g = w.g_mlp;
    a.rstd = act.at<float>(act.L.rstd2);
    a.gy = W(BL.gh);
    a.gres = ds.p;
    a.gres_f32 = ds.f32;
    a.res_map = {mv.idx, S};
    if (scatter) {
      a.gx = ds.p;
      a.gx_f32 = ds.f32;
      a.dst = {mv.idx, S};
    } else {
      a.gx = W(BL.gz32);
      a.gx_f32 = 1;
      a.dst = {nullptr, 1};
      a.gx2 = dt == LD_BF16 ? W(BL.gz) : nullptr;
    }
    a.dg_part = reinterpret_cast<float*>(ws + BL.dg_part);
    a.rc = {mv.count, S, T};
    a.d = static_cast<int32_t>(D.d);
    ProfScope ps("ld_rmsnorm_bwd_k", s);
    if ((e = launch_rmsnorm_bwd(dt, a, dw.g_mlp, s)) != hipSuccess) return fail(LD_E_HIP, "rmsnorm_bwd: %s", hipGetErrorString(e));
    const double res_es = ds.f32 ? 4.0 : D.es;
    const double out_es = scatter ? res_es : 4.0 + (a.gx2 ? D.es : 0.0);
    ps.end(0, (4.0 + D.es + res_es + out_es) * hm * D.d);
  }
  return LD_OK;
}

// Backward of attn_forward_part on the rows mv keeps; dL/dX^l of those rows
// is written into the gradient stream ds.  gather = 0 takes dL/dZ from the
// scratch (gz32 / gz, left by ffn_backward_part for the same rows); gather =
// 1 reads the kept rows of the stream, which then holds dL/dZ.
int attn_backward_part(const Dims& D, const ld_weights& w, const MaskView& mv, const ActPtrs& act,
                       const BwdLayout& BL, char* ws, Stream ds, const ld_grads& dw, int64_t hc,
                       bool gather, hipStream_t s) {
  const int dt = D.dtype;
  const int64_t T = D.T;
  const int64_t hm = hc * D.S;
  const int32_t S = static_cast<int32_t>(D.S);
  auto W = [&](size_t off) { return static_cast<void*>(ws + off); };
  float* SK = BL.splitk_bytes ? reinterpret_cast<float*>(ws + BL.splitk) : nullptr;
  hipError_t e;
  // the operand of the output projection's backward GEMMs: gz (bf16) or
  // gz32 (float32 configurations), gathered from the stream under sub-layer
  // granularity
  void* gz_op = dt == LD_BF16 ? W(BL.gz) : W(BL.gz32);
  if (gather) {
    RowsArgs a{};
    a.src = ds.p;
    a.src_f32 = ds.f32;
    a.dst = gz_op;
    a.src_map = {mv.idx, S};
    a.dst_map = {nullptr, 1};
    a.rc = {mv.count, S, T};
    a.d = static_cast<int32_t>(D.d);
    ProfScope ps("ld_gather_rows_k", s);
    if ((e = launch_gather(dt, a, s)) != hipSuccess) return fail(LD_E_HIP, "gather: %s", hipGetErrorString(e));
    ps.end(0, ((ds.f32 ? 4.0 : D.es) + D.es) * hm * D.d);
  }
  // ga = r * gz W_o [M, d] and dW_o = r * gz^T att [d, d]; gh1 = gqkv W_qkv
  // [M, d] and dW_qkv = gqkv^T h1 [3d, d].  With the 256x256 kernels dW_o
  // waits for the QKV launch, which then holds both weight gradients: ga
  // runs alone, and the two weight gradients (long workgroups) and gh1
  // (short ones) fill one launch, mostly without split-K.
  GemmArgs g_ga = gemm_args();
  g_ga.A = gz_op;
  g_ga.lda = D.d;
  g_ga.B = w.w_o;
  g_ga.ldb = D.d;
  g_ga.C = W(BL.ga);
  g_ga.ldc = D.d;
  g_ga.alpha_dev = mv.r;
  g_ga.N = static_cast<int32_t>(D.d);
  g_ga.K = static_cast<int32_t>(D.d);
  g_ga.dev_count = mv.count;
  g_ga.count_mult = S;
  GemmArgs g_wo = gemm_args();
  g_wo.A = gz_op;
  g_wo.lda = D.d;
  g_wo.B = act.at(act.L.att);
  g_wo.ldb = D.d;
  g_wo.C = dw.w_o;
  g_wo.ldc = D.d;
  g_wo.c_f32 = 1;
  g_wo.alpha_dev = mv.r;
  g_wo.M = static_cast<int32_t>(D.d);
  g_wo.N = static_cast<int32_t>(D.d);
  g_wo.dev_count = mv.count;
  g_wo.count_mult = S;
  g_wo.count_dim = 1;
  GemmArgs g_gh1 = gemm_args();
  g_gh1.A = W(BL.gqkv);
  g_gh1.lda = 3 * D.d;
  g_gh1.B = w.w_qkv;
  g_gh1.ldb = D.d;
  g_gh1.C = W(BL.gh);
  g_gh1.ldc = D.d;
  g_gh1.N = static_cast<int32_t>(D.d);
  g_gh1.K = static_cast<int32_t>(3 * D.d);
  g_gh1.dev_count = mv.count;
  g_gh1.count_mult = S;
  GemmArgs g_wqkv = gemm_args();
  g_wqkv.A = W(BL.gqkv);
  g_wqkv.lda = 3 * D.d;
  g_wqkv.B = act.at(act.L.h1);
  g_wqkv.ldb = D.d;
  g_wqkv.C = dw.w_qkv;
  g_wqkv.ldc = D.d;
  g_wqkv.c_f32 = 1;
  g_wqkv.M = static_cast<int32_t>(3 * D.d);
  g_wqkv.N = static_cast<int32_t>(D.d);
  g_wqkv.dev_count = mv.count;
  g_wqkv.count_mult = S;
  g_wqkv.count_dim = 1;
  const GemmArgs none = gemm_args();  // M = 0: no weight gradient in the launch
  const bool grouped = group_weight_grads(dt, g_wo, g_ga, g_wqkv, g_gh1, hm, T, SK != nullptr);
  if (int rc = run_gemm_pair(dt, grouped ? none : g_wo, hm, T, g_ga, T, hm, D.d, s, SK, BL.splitk_bytes)) return rc;
  // attention backward -> gqkv
  {
    AttnArgs a{};
    a.qkv = act.at(act.L.qkv);
    a.o = act.at(act.L.att);
    a.go = W(BL.ga);
    a.out = W(BL.gqkv);
    a.lse = act.at<float>(act.L.lse);
    a.delta = reinterpret_cast<float*>(ws + BL.delta);
    a.dev_count = mv.count;
    a.n_seq = static_cast<int32_t>(D.B);
    a.S = S;
    a.H = static_cast<int32_t>(D.H);
    a.dh = static_cast<int32_t>(D.dh);
    a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(D.dh)));
    a.alibi = D.kind == LD_BLOCK_ALIBI_RELU2;
    // algorithmic FLOPs of the backward (2x the forward), split over the two
    // MFMA kernels in proportion to the products each forms (dK/dV 4, dQ 3);
    // bytes: the delta kernel reads O and dO, the MFMA kernels five tensors
    // (the bf16 dQ kernel, which forms delta, also O)
    const double fl_bwd = 4.0 * hc * D.d * D.S * (D.S + 1.0);
    for (int part = 0; part < attn_bwd_parts(dt); ++part) {
      const char* name = attn_bwd_kernel_name(dt, part);
      const bool dkdv = std::strstr(name, "dkdv") != nullptr, dq = std::strstr(name, "_dq_") != nullptr;
      ProfScope ps(name, s);
      if ((e = launch_attn_bwd_part(dt, part, a, s)) != hipSuccess)
        return fail(LD_E_HIP, "attn_bwd: %s", hipGetErrorString(e));
      ps.end(dkdv ? fl_bwd * 4.0 / 7.0 : dq ? fl_bwd * 3.0 / 7.0 : 0.0,
             D.es * hm * D.d * (dkdv ? 5.0 : dq ? (dt == LD_BF16 ? 6.0 : 5.0) : 2.0));
    }
  }
  if (int rc = run_gemm_pair(dt, g_wqkv, hm, T, g_gh1, T, hm, 3 * D.d, s, SK, BL.splitk_bytes,
                             grouped ? &g_wo : nullptr))
    return rc;
  // dL/dX^l[kept rows] = dL/dZ + RMSNorm_bwd(xk, g_attn, gh1); dg_attn.  dL/dZ
  // is gz32 (float32), or the stream's rows under sub-layer granularity.
  {
    RmsBwdArgs a{};
    a.x = act.at(act.L.xk);
    a.x_f32 = 1;
    a.g = w.g_attn;
    a.rstd = act.at<float>(act.L.rstd1);
    a.gy = W(BL.gh);
    if (gather) {
      a.gres = ds.p;
      a.gres_f32 = ds.f32;
      a.res_map = {mv.idx, S};
    } else {
      a.gres = W(BL.gz32);
      a.gres_f32 = 1;
      a.res_map = {nullptr, 1};
    }
    a.gx = ds.p;
    a.gx_f32 = ds.f32;
    a.dst = {mv.idx, S};
    a.dg_part = reinterpret_cast<float*>(ws + BL.dg_part);
    a.rc = {mv.count, S, T};
    a.d = static_cast<int32_t>(D.d);
    ProfScope ps("ld_rmsnorm_bwd_k", s);
    if ((e = launch_rmsnorm_bwd(dt, a, dw.g_attn, s)) != hipSuccess) return fail(LD_E_HIP, "rmsnorm_bwd: %s", hipGetErrorString(e));
    const double st_es = ds.f32 ? 4.0 : D.es;
    ps.end(0, (4.0 + D.es + (gather ? st_es : 4.0) + st_es) * hm * D.d);
  }
  return LD_OK;
}

// One layer backward (FFN sub-block, then attention), mirroring layer_forward.
// A sub-block the host knows to be dropped for the whole batch launches only
// the zero fill of its weight gradients.
int layer_backward(const Dims& D, const ld_weights& w, const LayerMasks& lm, const ActPtrs& act,
                   const BwdLayout& BL, char* ws, Stream ds, const ld_grads& dw, hipStream_t s) {
  if (!D.sub) {
    if (lm.host_a == 0) return zero_grads(D, dw, true, true, s);
    if (int rc = ffn_backward_part(D, w, lm.a, act, BL, ws, ds, dw, lm.hc_a, false, s)) return rc;
    return attn_backward_part(D, w, lm.a, act, BL, ws, ds, dw, lm.hc_a, false, s);
  }
  if (lm.host_f == 0) {
    if (int rc = zero_grads(D, dw, false, true, s)) return rc;
  } else if (int rc = ffn_backward_part(D, w, lm.f, act, BL, ws, ds, dw, lm.hc_f, true, s)) {
    return rc;
  }
  if (lm.host_a == 0) return zero_grads(D, dw, true, false, s);
  return attn_backward_part(D, w, lm.a, act, BL, ws, ds, dw, lm.hc_a, true, s);
}

int check_weights(const ld_weights* w) {
  if (!w || !w->g_attn || !w->w_qkv || !w->w_o || !w->g_mlp || !w->w_gate_up || !w->w_down)
    return fail(LD_E_INVALID, "weights pointer NULL");
  return LD_OK;
}
int check_grads(const ld_grads* g) {
  if (!g || !g->g_attn || !g->w_qkv || !g->w_o || !g->g_mlp || !g->w_gate_up || !g->w_down)
    return fail(LD_E_INVALID, "grads pointer NULL");
  return LD_OK;
}

// nm masks per layer, drawn per sequence or (per_batch) once per layer.
int launch_mask_range(const ld_config* cfg, int32_t n, int32_t batch, int32_t nm, int32_t per_batch,
                      const float* p, int32_t first, uint64_t seed, uint64_t step, const uint8_t* ovr,
                      uint8_t* keep, int32_t* idx, int32_t* count, float* r_out, hipStream_t s) {
  for (int32_t l0 = 0; l0 < n; l0 += kMaxMaskLayers) {
    const int32_t nl = std::min<int32_t>(kMaxMaskLayers, n - l0);
    MaskArgs a;
    std::memset(&a, 0, sizeof(a));
    for (int32_t i = 0; i < nl; ++i) {
      threshold(p[l0 + i], &a.thr[i], &a.drop_all[i]);
      a.r[i] = cfg ? residual_scale(cfg, p[l0 + i]) : 0.f;
    }
    a.n_layers = nl;
    a.batch = batch;
    a.first_layer = first + l0;
    a.n_masks = nm;
    a.per_batch = per_batch;
    a.seed = seed;
    a.step = step;
    const int64_t rows = static_cast<int64_t>(l0) * nm;
    a.keep_override = ovr ? ovr + rows * batch : nullptr;
    a.keep = keep + rows * batch;
    a.idx = idx + rows * batch;
    a.count = count + rows;
    a.r_out = r_out ? r_out + l0 : nullptr;
    ProfScope ps("ld_mask_compact", s);
    hipError_t e = launch_masks(a, s);
    if (e != hipSuccess) return fail(LD_E_HIP, "mask launch: %s", hipGetErrorString(e));
    ps.end(0, 13.0 * nl * nm * batch);
  }
  return LD_OK;
}

// What the host knows of mask m of `layer` before any launch: under per-batch
// granularity without an override the draw is taken here (the same Philox
// block the mask kernel uses), so 0 = dropped for the whole batch and 1 =
// kept; -1 otherwise (decided on the device).
int host_mask_state(const Dims& D, float p, int64_t layer, uint64_t seed, uint64_t step,
                    const uint8_t* ovr, int m) {
  if (!D.per_batch || ovr) return -1;
  uint64_t thr;
  uint8_t drop_all;
  threshold(p, &thr, &drop_all);
  if (drop_all) return 0;
  return mask_draw(0, static_cast<uint64_t>(layer), step, seed, 1, m) < thr ? 0 : 1;
}

// Kept count of mask m of `layer`, from the mask kernel's own draws taken
// again on the host (B Philox blocks), or -1 when an override decides.
int64_t host_kept_count(const Dims& D, float p, int64_t layer, uint64_t seed, uint64_t step, const uint8_t* ovr,
                        int m) {
  if (ovr) return -1;
  uint64_t thr;
  uint8_t drop_all;
  threshold(p, &thr, &drop_all);
  if (drop_all) return 0;
  int64_t kept = 0;
  for (int64_t b = 0; b < D.B; ++b)
    kept += mask_draw(static_cast<uint64_t>(b), static_cast<uint64_t>(layer), step, seed, D.per_batch, m) < thr ? 0 : 1;
  return kept;
}

// The masks of layer l of a block laid out by mask_layout (layer-major).
// draws: p, seed and step are the ones the mask kernel draws with, so the
// host knows the kept counts (the device still decides every row; the
// counts only plan launches and skip a sub-block no sample keeps).
LayerMasks layer_masks(const Dims& D, const MaskLayout& ml, char* base, int64_t l, int64_t layer_id,
                       float p, uint64_t seed, uint64_t step, const uint8_t* ovr,
                       const std::vector<int64_t>& hc, bool draws = true) {
  uint8_t* keep = reinterpret_cast<uint8_t*>(base + ml.keep);
  int32_t* idx = reinterpret_cast<int32_t*>(base + ml.idx);
  int32_t* count = reinterpret_cast<int32_t*>(base + ml.count);
  float* r = reinterpret_cast<float*>(base + ml.r);
  auto view = [&](int64_t m) {
    const int64_t row = l * D.nm + m;
    return MaskView{keep + row * D.B, idx + row * D.B, count + row, r + l};
  };
  LayerMasks lm{};
  lm.a = view(0);
  lm.f = view(D.nm - 1);
  lm.host_a = host_mask_state(D, p, layer_id, seed, step, ovr, 0);
  lm.host_f = host_mask_state(D, p, layer_id, seed, step, ovr, D.nm - 1);
  lm.hc_a = hc[l * D.nm];
  lm.hc_f = hc[l * D.nm + D.nm - 1];
  if (draws && !ovr) {
    lm.hc_a = host_kept_count(D, p, layer_id, seed, step, ovr, 0);
    lm.hc_f = D.nm > 1 ? host_kept_count(D, p, layer_id, seed, step, ovr, D.nm - 1) : lm.hc_a;
    if (lm.hc_a == 0) lm.host_a = 0;
    if (lm.hc_f == 0) lm.host_f = 0;
  }
  return lm;
}

// When the device counts were read back (profiling), the host's own counts
// must equal them: they plan the launches and skip sub-blocks.
int check_host_counts(const Dims& D, const LayerMasks& lm, const std::vector<int64_t>& hc, int64_t l) {
  const int64_t da = hc[l * D.nm], df = hc[l * D.nm + D.nm - 1];
  if ((da >= 0 && lm.hc_a >= 0 && da != lm.hc_a) || (df >= 0 && lm.hc_f >= 0 && df != lm.hc_f))
    return fail(LD_E_HIP, "layer %lld: device kept counts %lld/%lld, host %lld/%lld", static_cast<long long>(l),
                static_cast<long long>(da), static_cast<long long>(df), static_cast<long long>(lm.hc_a),
                static_cast<long long>(lm.hc_f));
  return LD_OK;
}

// ------------------------------------------------------ decoding helpers

// Scratch of ld_stack_decode for n_new rows per sequence and caches of s_max
// positions.
struct DecLayout {
  size_t h, rstd, qkv, att, z, uv, s, part_o, part_ml, skp, skp_bytes, total;
};

size_t skinny_part_bytes(int64_t M, int64_t N, int64_t K) {
  if (M > kSkinnyMaxM) return 0;
  const int ks = skinny_ksplit(M, N, K);
  return ks > 1 ? static_cast<size_t>(ks) * M * N * 4 : 0;
}

// Partials of a skinny GEMM whose reduction is fused with what follows it
// (written even with one split).
size_t skinny_fused_part_bytes(int64_t M, int64_t N, int64_t K) {
  if (M > kSkinnyMaxM) return 0;
  return static_cast<size_t>(skinny_ksplit(M, N, K)) * M * N * 4;
}


int64_t dec_chunks(int64_t keys) { return (keys + kDecKeys - 1) / kDecKeys; }

DecLayout dec_layout(const Dims& D, int64_t n_new, int64_t s_max) {
  DecLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += up(bytes);
    return at;
  };
  const size_t es = D.es, M = D.B * n_new;
  L.h = take(es * M * D.d);
  L.rstd = take(4 * M);
  L.qkv = take(es * M * 3 * D.d);
  L.att = take(es * M * D.d);
  L.z = take(es * M * D.d);
  L.uv = take(es * M * D.fw);
  L.s = take(es * M * D.f);
  const size_t pc = static_cast<size_t>(D.B) * D.H * dec_chunks(s_max) * kDecMaxRows;
  L.part_o = take(4 * pc * D.dh);
  L.part_ml = take(4 * pc * 2);
  const int64_t shapes[4][2] = {{3 * D.d, D.d}, {D.d, D.d}, {D.fw, D.d}, {D.d, D.f}};
  for (const auto& sh : shapes) L.skp_bytes = std::max(L.skp_bytes, skinny_fused_part_bytes(M, sh[0], sh[1]));
  L.skp = take(L.skp_bytes);
  L.total = o;
  return L;
}

// Where a qkv projection's keys/values also go (see SkinnyArgs).
struct KvOut {
  void* kv;
  int32_t d, n, s_max, pos;
};

// C[M, N] = (R ? R : 0) + alpha * A W^T for the rows of a decoding step:
// the skinny kernel for M <= kSkinnyMaxM, else the general GEMM.  kv: the
// columns from kv.d on also go to that cache (skinny kernel), or the caller
// stores them (general GEMM: returns with *kv_done = false).
int dec_gemm(const void* A, int64_t lda, const void* W, int64_t ldw, void* C, int64_t ldc,
             const void* R, int64_t ldr, int64_t M, int64_t N, int64_t K, float alpha, float* part,
             size_t part_bytes, hipStream_t s, const KvOut* kv = nullptr, bool* kv_done = nullptr) {
  if (kv_done) *kv_done = false;
  if (M > kSkinnyMaxM) {
    GemmArgs g = gemm_args();
    g.A = A;
    g.lda = lda;
    g.B = W;
    g.ldb = ldw;
    g.C = C;
    g.ldc = ldc;
    g.R = R;
    g.ldr = ldr;
    g.M = static_cast<int32_t>(M);
    g.N = static_cast<int32_t>(N);
    g.K = static_cast<int32_t>(K);
    g.alpha = alpha;
    return run_gemm(LD_BF16, 1, 1, g, M, M, K, s);
  }
  SkinnyArgs g{};
  g.A = A;
  g.lda = lda;
  g.W = W;
  g.ldw = ldw;
  g.C = C;
  g.ldc = ldc;
  g.R = R;
  g.ldr = ldr;
  g.M = static_cast<int32_t>(M);
  g.N = static_cast<int32_t>(N);
  g.K = static_cast<int32_t>(K);
  g.alpha = alpha;
  const int ks = skinny_ksplit(M, N, K);
  if (ks > 1) {
    if (static_cast<size_t>(ks) * M * N * 4 > part_bytes) return fail(LD_E_WORKSPACE, "skinny GEMM scratch too small");
    g.part = part;
  }
  if (kv) {
    g.kv = kv->kv;
    g.kv_d = kv->d;
    g.kv_n = kv->n;
    g.kv_s_max = kv->s_max;
    g.kv_pos = kv->pos;
    if (kv_done) *kv_done = true;
  }
  ProfScope ps(M <= 32 ? "ld_gemm_bf16_skinny<1>" : "ld_gemm_bf16_skinny<2>", s);
  hipError_t e = launch_gemm_skinny(g, ks, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "skinny GEMM: %s", hipGetErrorString(e));
  ps.end(2.0 * M * N * K, 2.0 * (M * K + N * K + M * N) + (R ? 2.0 * M * N : 0.0));
  return LD_OK;
}

// Fused decode projection (at most 8 rows; see launch_gemm_dec): C = act(R +
// alpha * A' W^T) with A' the RMSNorm of A's rows when g is set.
int dec_proj(const void* A, int64_t lda, const void* g, float eps, const void* W, int64_t ldw, void* C,
             int64_t ldc, const void* R, int64_t ldr, int64_t M, int64_t N, int64_t K, float alpha, int act,
             hipStream_t s, const KvOut* kv = nullptr) {
  SkinnyArgs a{};
  a.A = A;
  a.lda = lda;
  a.W = W;
  a.ldw = ldw;
  a.C = C;
  a.ldc = ldc;
  a.R = R;
  a.ldr = ldr;
  a.M = static_cast<int32_t>(M);
  a.N = static_cast<int32_t>(N);
  a.K = static_cast<int32_t>(K);
  a.alpha = alpha;
  a.g = g;
  a.eps = eps;
  a.act = act;
  if (kv) {
    a.kv = kv->kv;
    a.kv_d = kv->d;
    a.kv_n = kv->n;
    a.kv_s_max = kv->s_max;
    a.kv_pos = kv->pos;
  }
  ProfScope ps("ld_gemm_bf16_dec", s);
  hipError_t e = launch_gemm_dec(a, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "decode projection: %s", hipGetErrorString(e));
  const double wrows = act == kDecActSwiglu ? 2.0 * N : static_cast<double>(N);
  ps.end(2.0 * M * wrows * K, 2.0 * (M * K + wrows * K + M * N) + (R ? 2.0 * M * N : 0.0));
  return LD_OK;
}

// Skinny GEMM (at most 64 rows) writing only its split-K partials, for a
// fused reduction launched next; g and ks describe them.
int skinny_part(const void* A, int64_t lda, const void* W, int64_t ldw, int64_t M, int64_t N, int64_t K,
                float alpha, float* part, size_t part_bytes, hipStream_t s, SkinnyArgs& g, int& ks) {
  g = SkinnyArgs{};
  g.A = A;
  g.lda = lda;
  g.W = W;
  g.ldw = ldw;
  g.M = static_cast<int32_t>(M);
  g.N = static_cast<int32_t>(N);
  g.K = static_cast<int32_t>(K);
  g.alpha = alpha;
  g.part = part;
  g.part_only = 1;
  ks = skinny_ksplit(M, N, K);
  if (static_cast<size_t>(ks) * M * N * 4 > part_bytes) return fail(LD_E_WORKSPACE, "skinny GEMM scratch too small");
  ProfScope ps(M <= 32 ? "ld_gemm_bf16_skinny<1>" : "ld_gemm_bf16_skinny<2>", s);
  const hipError_t e = launch_gemm_skinny(g, ks, s);
  if (e != hipSuccess) return fail(LD_E_HIP, "skinny GEMM: %s", hipGetErrorString(e));
  ps.end(2.0 * M * N * K, 2.0 * (M * K + N * K) + 4.0 * ks * M * N);
  return LD_OK;
}

}  // namespace

// ====================================================================== ABI

extern "C" {

const char* ld_status_string(int status) {
  switch (status) {
    case LD_OK: return "LD_OK";
    case LD_E_INVALID: return "LD_E_INVALID";
    case LD_E_SHAPE: return "LD_E_SHAPE";
    case LD_E_UNSUPPORTED: return "LD_E_UNSUPPORTED";
    case LD_E_WORKSPACE: return "LD_E_WORKSPACE";
    case LD_E_HIP: return "LD_E_HIP";
  }
  return "LD_E_UNKNOWN";
}

const char* ld_last_error(void) { return t_err.c_str(); }

int ld_schedule_p(int32_t dist, int32_t sched, float p_max, int32_t layer, int32_t n_layers,
                  int64_t t, int64_t n_steps, float* p_out) {
  t_err.clear();
  if (!p_out) return fail(LD_E_INVALID, "p_out is NULL");
  if (std::isnan(p_max) || p_max < 0.f || p_max > 1.f) return fail(LD_E_INVALID, "p_max outside [0, 1]");
  if (n_layers < 1 || layer < 0 || layer >= n_layers) return fail(LD_E_INVALID, "layer outside [0, n_layers)");
  if (n_steps < 1) return fail(LD_E_INVALID, "n_steps < 1");
  double depth;
  switch (dist) {
    case 0: depth = p_max; break;
    case 1: depth = n_layers == 1 ? 0.0 : static_cast<double>(layer) / (n_layers - 1) * p_max; break;
    case 2: depth = (layer % 2 == 1) ? static_cast<double>(p_max) : 0.0; break;
    default: return fail(LD_E_INVALID, "unknown distribution %d", dist);
  }
  double tf;
  const int64_t tc = std::min<int64_t>(std::max<int64_t>(t, 0), n_steps - 1);
  const double frac = n_steps <= 1 ? 0.0 : static_cast<double>(tc) / static_cast<double>(n_steps - 1);
  switch (sched) {
    case 0: tf = 1.0; break;
    case 1: tf = frac; break;
    case 2: tf = 1.0 - frac; break;
    default: return fail(LD_E_INVALID, "unknown schedule %d", sched);
  }
  *p_out = static_cast<float>(depth * tf);
  return LD_OK;
}

int ld_masks(int32_t n_layers, int32_t batch, const float* p, int32_t first_layer, uint64_t seed,
             uint64_t step, uint8_t* keep, int32_t* idx, int32_t* count, void* stream) {
  return ld_masks_granular(LD_GRAN_LAYER_SEQ, n_layers, batch, p, first_layer, seed, step, keep, idx,
                           count, stream);
}

int ld_masks_granular(int32_t granularity, int32_t n_layers, int32_t batch, const float* p,
                      int32_t first_layer, uint64_t seed, uint64_t step, uint8_t* keep, int32_t* idx,
                      int32_t* count, void* stream) {
  t_err.clear();
  if (granularity < 0 || granularity > 3) return fail(LD_E_INVALID, "unknown granularity %d", granularity);
  if (n_layers < 1 || n_layers > kMaxMaskLayers) return fail(LD_E_INVALID, "n_layers outside [1, %d]", kMaxMaskLayers);
  if (batch < 1) return fail(LD_E_INVALID, "batch < 1");
  if (first_layer < 0) return fail(LD_E_INVALID, "first_layer < 0");
  if (!p || !keep || !idx || !count) return fail(LD_E_INVALID, "NULL pointer");
  for (int32_t i = 0; i < n_layers; ++i)
    if (int rc = check_p(p[i])) return rc;
  const int32_t nm = granularity & LD_GRAN_SUBLAYER ? 2 : 1;
  const int32_t pb = granularity & LD_GRAN_PER_BATCH ? 1 : 0;
  return launch_mask_range(nullptr, n_layers, batch, nm, pb, p, first_layer, seed, step, nullptr, keep,
                           idx, count, nullptr, as_stream(stream));
}

int ld_gather_rows(const ld_config* cfg, const int32_t* idx, const int32_t* count, const void* x,
                   void* xk, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (!idx || !count || !x || !xk) return fail(LD_E_INVALID, "NULL pointer");
  RowsArgs a{};
  a.src = x;
  a.dst = xk;
  a.src_map = {idx, static_cast<int32_t>(D.S)};
  a.dst_map = {nullptr, 1};
  a.rc = {count, static_cast<int32_t>(D.S), D.T};
  a.d = static_cast<int32_t>(D.d);
  hipError_t e = launch_gather(D.dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "gather: %s", hipGetErrorString(e));
  return LD_OK;
}

int ld_scatter_add_rows(const ld_config* cfg, const int32_t* idx, const int32_t* count, float r,
                        const void* yk, void* x, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (!idx || !count || !x || !yk) return fail(LD_E_INVALID, "NULL pointer");
  if (!std::isfinite(r)) return fail(LD_E_INVALID, "r not finite");
  RowsArgs a{};
  a.src = yk;
  a.dst = x;
  a.src_map = {nullptr, 1};
  a.dst_map = {idx, static_cast<int32_t>(D.S)};
  a.rc = {count, static_cast<int32_t>(D.S), D.T};
  a.d = static_cast<int32_t>(D.d);
  a.r = r;
  hipError_t e = launch_scatter_add(D.dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "scatter_add: %s", hipGetErrorString(e));
  return LD_OK;
}

size_t ld_layer_ctx_bytes(const ld_config* cfg) {
  Dims D;
  if (check_cfg(cfg, &D)) return 0;
  return mask_layout(1, D.B, D.nm).total + act_layout(D).total;
}

size_t ld_layer_ws_bytes(const ld_config* cfg) {
  Dims D;
  if (check_cfg(cfg, &D)) return 0;
  return bwd_layout(D).total;
}

// Bytes of the float32 copies of x and dx that ld_stack_step keeps in its
// workspace (bf16 configurations; float32 ones run on the caller's tensors).
size_t stream_bytes(const Dims& D) { return D.dtype == LD_BF16 ? up(4ull * D.T * D.d) : 0; }

size_t ld_stack_ws_bytes(const ld_config* cfg, int32_t n_layers) {
  Dims D;
  if (check_cfg(cfg, &D) || n_layers < 1) return 0;
  return mask_layout(n_layers, D.B, D.nm).total + static_cast<size_t>(n_layers) * act_layout(D).total +
         bwd_layout(D).total + 2 * stream_bytes(D);
}

int ld_layer_fwd(const ld_config* cfg, const ld_weights* w, int32_t layer, float p, uint64_t seed,
                 uint64_t step, void* x, void* ctx, void* ws, size_t ws_bytes,
                 const uint8_t* keep_override, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (int rc = check_weights(w)) return rc;
  if (int rc = check_p(p)) return rc;
  if (layer < 0) return fail(LD_E_INVALID, "layer < 0");
  if (!x || !ctx) return fail(LD_E_INVALID, "NULL pointer");
  (void)ws;
  (void)ws_bytes;
  hipStream_t s = as_stream(stream);
  const MaskLayout ml = mask_layout(1, D.B, D.nm);
  char* c = static_cast<char*>(ctx);
  int32_t* count = reinterpret_cast<int32_t*>(c + ml.count);
  if (int rc = launch_mask_range(cfg, 1, static_cast<int32_t>(D.B), D.nm, D.per_batch, &p, layer, seed,
                                 step, keep_override, reinterpret_cast<uint8_t*>(c + ml.keep),
                                 reinterpret_cast<int32_t*>(c + ml.idx), count,
                                 reinterpret_cast<float*>(c + ml.r), s))
    return rc;
  ActPtrs act{c + ml.total, act_layout(D)};
  const std::vector<int64_t> hc = host_counts_if_profiling(count, D.nm, s);
  const LayerMasks lm = layer_masks(D, ml, c, 0, layer, p, seed, step, keep_override, hc);
  if (int rc = check_host_counts(D, lm, hc, 0)) return rc;
  return layer_forward(cfg, D, *w, lm, act, Stream{x, D.dtype == LD_F32}, s);
}

int ld_layer_bwd(const ld_config* cfg, const ld_weights* w, const void* ctx, void* dx,
                 const ld_grads* dw, void* ws, size_t ws_bytes, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (int rc = check_weights(w)) return rc;
  if (int rc = check_grads(dw)) return rc;
  if (!ctx || !dx || !ws) return fail(LD_E_INVALID, "NULL pointer");
  const BwdLayout BL = bwd_layout(D);
  if (ws_bytes < BL.total) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, BL.total);
  const MaskLayout ml = mask_layout(1, D.B, D.nm);
  char* c = const_cast<char*>(static_cast<const char*>(ctx));
  ActPtrs act{c + ml.total, act_layout(D)};
  hipStream_t s = as_stream(stream);
  const std::vector<int64_t> hc =
      host_counts_if_profiling(reinterpret_cast<int32_t*>(c + ml.count), D.nm, s);
  // the ctx carries no p, seed or step: every decision is the device's
  LayerMasks lm = layer_masks(D, ml, c, 0, 0, 0.f, 0, 0, nullptr, hc, false);
  lm.host_a = lm.host_f = -1;
  return layer_backward(D, *w, lm, act, BL, static_cast<char*>(ws), Stream{dx, D.dtype == LD_F32}, *dw, s);
}

int ld_stack_step(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const float* p,
                  uint64_t seed, uint64_t step, void* x, void* dx, const ld_grads* dw, void* ws,
                  size_t ws_bytes, const uint8_t* keep_override, uint8_t* keep_out,
                  int32_t* idx_out, int32_t* count_out, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (n_layers < 1 || n_layers > 1024) return fail(LD_E_INVALID, "n_layers outside [1, 1024]");
  if (!w || !p || !dw || !x || !dx || !ws) return fail(LD_E_INVALID, "NULL pointer");
  for (int32_t l = 0; l < n_layers; ++l) {
    if (int rc = check_weights(&w[l])) return rc;
    if (int rc = check_grads(&dw[l])) return rc;
    if (int rc = check_p(p[l])) return rc;
  }
  const size_t need = ld_stack_ws_bytes(cfg, n_layers);
  if (ws_bytes < need) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = as_stream(stream);
  const int64_t L = n_layers, B = D.B;
  const int64_t nm = D.nm;
  const MaskLayout ml = mask_layout(L, B, nm);
  const ActLayout al = act_layout(D);
  const BwdLayout BL = bwd_layout(D);
  char* base = static_cast<char*>(ws);
  uint8_t* keep = reinterpret_cast<uint8_t*>(base + ml.keep);
  int32_t* idx = reinterpret_cast<int32_t*>(base + ml.idx);
  int32_t* count = reinterpret_cast<int32_t*>(base + ml.count);
  char* acts = base + ml.total;
  char* bws = acts + static_cast<size_t>(L) * al.total;
  // bf16 configurations: the residual streams in float32 for the whole step
  const bool cp = D.dtype == LD_BF16;
  const Stream xs{cp ? bws + BL.total : x, 1};
  const Stream dxs{cp ? bws + BL.total + stream_bytes(D) : dx, 1};
  const int64_t n_elems = D.T * D.d;

  if (int rc = launch_mask_range(cfg, n_layers, static_cast<int32_t>(B), D.nm, D.per_batch, p, 0, seed,
                                 step, keep_override, keep, idx, count,
                                 reinterpret_cast<float*>(base + ml.r), s))
    return rc;
  const std::vector<int64_t> hc = host_counts_if_profiling(count, L * nm, s);
  std::vector<LayerMasks> lms;
  lms.reserve(L);
  for (int64_t l = 0; l < L; ++l) lms.push_back(layer_masks(D, ml, base, l, l, p[l], seed, step, keep_override, hc));
  for (int64_t l = 0; l < L; ++l)
    if (int rc = check_host_counts(D, lms[l], hc, l)) return rc;
  auto convert = [&](const void* src, void* dst, int to_f32) {
    ProfScope ps("ld_convert_k", s);
    const hipError_t e = launch_convert(src, dst, n_elems, to_f32, s);
    if (e != hipSuccess) return fail(LD_E_HIP, "convert: %s", hipGetErrorString(e));
    ps.end(0, 6.0 * n_elems);
    return static_cast<int>(LD_OK);
  };
  if (cp)
    if (int rc = convert(x, xs.p, 1)) return rc;
  for (int64_t l = 0; l < L; ++l) {
    ActPtrs act{acts + static_cast<size_t>(l) * al.total, al};
    if (int rc = layer_forward(cfg, D, w[l], lms[l], act, xs, s)) return rc;
  }
  if (cp) {
    if (int rc = convert(xs.p, x, 0)) return rc;
    if (int rc = convert(dx, dxs.p, 1)) return rc;
  }
  for (int64_t l = L - 1; l >= 0; --l) {
    ActPtrs act{acts + static_cast<size_t>(l) * al.total, al};
    if (int rc = layer_backward(D, w[l], lms[l], act, BL, bws, dxs, dw[l], s)) return rc;
  }
  if (cp)
    if (int rc = convert(dxs.p, dx, 0)) return rc;
  if (keep_out) LD_HIP(hipMemcpyAsync(keep_out, keep, L * nm * B, hipMemcpyDeviceToDevice, s));
  if (idx_out) LD_HIP(hipMemcpyAsync(idx_out, idx, 4 * L * nm * B, hipMemcpyDeviceToDevice, s));
  if (count_out) LD_HIP(hipMemcpyAsync(count_out, count, 4 * L * nm, hipMemcpyDeviceToDevice, s));
  return LD_OK;
}

// ------------------------------------------------ evaluation and decoding

size_t ld_eval_ws_bytes(const ld_config* cfg) {
  Dims D;
  if (check_cfg(cfg, &D)) return 0;
  return act_layout(D).total;
}

int ld_stack_eval(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const uint8_t* active,
                  const float* r_eval, void* x, void* const* kv, int32_t s_max, void* ws,
                  size_t ws_bytes, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (n_layers < 1 || n_layers > 1024) return fail(LD_E_INVALID, "n_layers outside [1, 1024]");
  if (!w || !x || !ws) return fail(LD_E_INVALID, "NULL pointer");
  if (kv && D.dtype != LD_BF16) return fail(LD_E_UNSUPPORTED, "KV caches are bf16 only");
  if (kv && s_max < D.S) return fail(LD_E_SHAPE, "s_max %d < seq %lld", s_max, static_cast<long long>(D.S));
  for (int32_t l = 0; l < n_layers; ++l) {
    if (active && !active[l]) continue;
    if (int rc = check_weights(&w[l])) return rc;
    if (r_eval && !std::isfinite(r_eval[l])) return fail(LD_E_INVALID, "r_eval[%d] not finite", l);
    if (kv && !kv[l]) return fail(LD_E_INVALID, "kv[%d] is NULL for an active layer", l);
  }
  const ActLayout al = act_layout(D);
  if (ws_bytes < al.total) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, al.total);
  hipStream_t s = as_stream(stream);
  ActPtrs act{static_cast<char*>(ws), al};
  for (int32_t l = 0; l < n_layers; ++l) {
    if (active && !active[l]) continue;
    MaskView mv{nullptr, nullptr, nullptr, nullptr, r_eval ? r_eval[l] : 1.f};
    const Stream xs{x, D.dtype == LD_F32};
    if (int rc = attn_forward_part(cfg, D, w[l], mv, act, xs, D.B, false, s, kv ? kv[l] : nullptr, s_max))
      return rc;
    if (int rc = ffn_forward_part(cfg, D, w[l], mv, act, xs, D.B, false, s)) return rc;
  }
  return LD_OK;
}

size_t ld_decode_ws_bytes(const ld_config* cfg, int32_t n_new, int32_t s_max) {
  Dims D;
  if (check_cfg(cfg, &D) || n_new < 1 || n_new > kDecMaxRows || s_max < 1) return 0;
  return dec_layout(D, n_new, s_max).total;
}

int ld_stack_decode(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const uint8_t* active,
                    const float* r_eval, void* x, void* const* kv, int32_t s_max, int32_t pos,
                    int32_t n_new, void* ws, size_t ws_bytes, void* stream) {
  t_err.clear();
  Dims D;
  if (int rc = check_cfg(cfg, &D)) return rc;
  if (D.dtype != LD_BF16) return fail(LD_E_UNSUPPORTED, "decoding is bf16 only");
  if (n_layers < 1 || n_layers > 1024) return fail(LD_E_INVALID, "n_layers outside [1, 1024]");
  if (!w || !x || !kv || !ws) return fail(LD_E_INVALID, "NULL pointer");
  if (n_new < 1 || n_new > kDecMaxRows) return fail(LD_E_INVALID, "n_new outside [1, %d]", kDecMaxRows);
  if (pos < 0 || s_max < 1 || static_cast<int64_t>(pos) + n_new > s_max)
    return fail(LD_E_SHAPE, "positions %d..%d outside the cache of %d", pos, pos + n_new - 1, s_max);
  for (int32_t l = 0; l < n_layers; ++l) {
    if (active && !active[l]) continue;
    if (int rc = check_weights(&w[l])) return rc;
    if (r_eval && !std::isfinite(r_eval[l])) return fail(LD_E_INVALID, "r_eval[%d] not finite", l);
    if (!kv[l]) return fail(LD_E_INVALID, "kv[%d] is NULL for an active layer", l);
  }
  const DecLayout L = dec_layout(D, n_new, s_max);
  if (ws_bytes < L.total) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);
  hipStream_t s = as_stream(stream);
  char* base = static_cast<char*>(ws);
  auto P = [&](size_t off) { return static_cast<void*>(base + off); };
  float* skp = L.skp_bytes ? reinterpret_cast<float*>(base + L.skp) : nullptr;
  const int64_t M = D.B * n_new, d = D.d;
  hipError_t e;
  auto norm = [&](const void* src, const void* gain) {
    RmsFwdArgs a{};
    a.x = src;
    a.src = {nullptr, 1};
    a.g = gain;
    a.y = P(L.h);
    a.rstd = reinterpret_cast<float*>(base + L.rstd);
    a.rc = {nullptr, 1, M};
    a.d = static_cast<int32_t>(d);
    a.eps = cfg->rms_eps;
    ProfScope ps("ld_rmsnorm_fwd_k", s);
    if ((e = launch_rmsnorm_fwd(LD_BF16, a, s)) != hipSuccess) return fail(LD_E_HIP, "rmsnorm_fwd: %s", hipGetErrorString(e));
    ps.end(0, 4.0 * M * d);
    return static_cast<int>(LD_OK);
  };
  // At most 8 rows (one new row per sequence of a batch of 8): each
  // projection is one fused launch that normalises its input rows and
  // applies the FFN activation itself.
  const bool fused = dec_gemm_ok(M, d, true) && dec_gemm_ok(M, D.f, false);
  // 9 to 64 rows (verify steps): split-K skinny GEMMs whose partial sums are
  // reduced together with what follows them: the residual and the next
  // RMSNorm (output and down projections), or the FFN activation.
  const bool part_fused = !fused && M <= kSkinnyMaxM;
  bool h_ready = false;  // L.h holds RMSNorm(x) with this layer's gain
  const int act = D.kind == LD_BLOCK_SWIGLU ? kDecActSwiglu : kDecActRelu2;
  for (int32_t l = 0; l < n_layers; ++l) {
    if (active && !active[l]) continue;
    const float r = r_eval ? r_eval[l] : 1.f;
    const ld_weights& wl = w[l];
    // h = RMSNorm(x); qkv = h W_qkv^T; new keys/values into the cache
    const KvOut ko{kv[l], static_cast<int32_t>(d), n_new, s_max, pos};
    bool kv_done = false;
    if (fused) {
      if (int rc = dec_proj(x, d, wl.g_attn, cfg->rms_eps, wl.w_qkv, d, P(L.qkv), 3 * d, nullptr, 0, M, 3 * d, d,
                            1.f, kDecActNone, s, &ko))
        return rc;
      kv_done = true;
    } else {
      if (!h_ready)
        if (int rc = norm(x, wl.g_attn)) return rc;
      h_ready = false;
      if (int rc = dec_gemm(P(L.h), d, wl.w_qkv, d, P(L.qkv), 3 * d, nullptr, 0, M, 3 * d, d, 1.f, skp,
                            L.skp_bytes, s, &ko, &kv_done))
        return rc;
    }
    if (!kv_done) {
      KvArgs k{};
      k.qkv = P(L.qkv);
      k.ld_qkv = 3 * d;
      k.cache = kv[l];
      k.s_max = s_max;
      k.d = static_cast<int32_t>(d);
      k.n = n_new;
      k.n_seq = static_cast<int32_t>(D.B);
      k.pos = pos;
      ProfScope ps("ld_kv_store_k", s);
      if ((e = launch_kv_store(k, s)) != hipSuccess) return fail(LD_E_HIP, "kv store: %s", hipGetErrorString(e));
      ps.end(0, 8.0 * M * d);
    }
    // attention of the new rows over positions 0..pos+n_new-1 of the cache
    DecAttnArgs at{};
    at.qkv = P(L.qkv);
    at.ld_qkv = 3 * d;
    at.cache = kv[l];
    at.s_max = s_max;
    at.out = P(L.att);
    at.part_o = reinterpret_cast<float*>(base + L.part_o);
    at.part_ml = reinterpret_cast<float*>(base + L.part_ml);
    at.n_seq = static_cast<int32_t>(D.B);
    at.H = static_cast<int32_t>(D.H);
    at.dh = static_cast<int32_t>(D.dh);
    at.n_new = n_new;
    at.pos = pos;
    at.n_chunks = static_cast<int32_t>(dec_chunks(static_cast<int64_t>(pos) + n_new));
    at.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(D.dh)));
    at.alibi = D.kind == LD_BLOCK_ALIBI_RELU2;
    {
      ProfScope ps("ld_attn_decode_bf16", s);
      if ((e = launch_attn_decode(at, s)) != hipSuccess) return fail(LD_E_HIP, "attn decode: %s", hipGetErrorString(e));
      const double keys = static_cast<double>(pos) + n_new;
      ps.end(4.0 * M * d * keys, 2.0 * D.B * keys * 2 * d + 4.0 * M * d);
    }
    // z = x + r (att W_o^T); h = RMSNorm(z); uv = h W_gate_up^T; s = act(uv)
    if (fused) {
      if (int rc = dec_proj(P(L.att), d, nullptr, 0.f, wl.w_o, d, P(L.z), d, x, d, M, d, d, r, kDecActNone, s))
        return rc;
      if (int rc = dec_proj(P(L.z), d, wl.g_mlp, cfg->rms_eps, wl.w_gate_up, d, P(L.s), D.f, nullptr, 0, M, D.f,
                            d, 1.f, act, s))
        return rc;
      // x = z + r (s W_down^T)
      if (int rc = dec_proj(P(L.s), D.f, nullptr, 0.f, wl.w_down, D.f, x, d, P(L.z), d, M, d, D.f, r,
                            kDecActNone, s))
        return rc;
      continue;
    }
    if (part_fused) {
      SkinnyArgs g{};
      int ks = 1;
      // z = x + r (att W_o^T) and h = RMSNorm(z)
      if (int rc = skinny_part(P(L.att), d, wl.w_o, d, M, d, d, r, skp, L.skp_bytes, s, g, ks)) return rc;
      g.C = P(L.z);
      g.ldc = d;
      g.R = x;
      g.ldr = d;
      if ((e = launch_skinny_reduce_norm(g, ks, wl.g_mlp, cfg->rms_eps, P(L.h), s)) != hipSuccess)
        return fail(LD_E_HIP, "skinny reduce: %s", hipGetErrorString(e));
      // s = act(h W_gate_up^T)
      if (int rc = skinny_part(P(L.h), d, wl.w_gate_up, d, M, D.fw, d, 1.f, skp, L.skp_bytes, s, g, ks)) return rc;
      if ((e = launch_skinny_reduce_act(g, ks, act, static_cast<int>(D.f), P(L.s), s)) != hipSuccess)
        return fail(LD_E_HIP, "skinny reduce: %s", hipGetErrorString(e));
      // x = z + r (s W_down^T), and the next active layer's h = RMSNorm(x)
      if (int rc = skinny_part(P(L.s), D.f, wl.w_down, D.f, M, d, D.f, r, skp, L.skp_bytes, s, g, ks)) return rc;
      g.C = x;
      g.ldc = d;
      g.R = P(L.z);
      g.ldr = d;
      int32_t next = l + 1;
      while (next < n_layers && active && !active[next]) ++next;
      const void* gain = next < n_layers ? w[next].g_attn : nullptr;
      if ((e = launch_skinny_reduce_norm(g, ks, gain, cfg->rms_eps, P(L.h), s)) != hipSuccess)
        return fail(LD_E_HIP, "skinny reduce: %s", hipGetErrorString(e));
      h_ready = gain != nullptr;
      continue;
    }
    if (int rc = dec_gemm(P(L.att), d, wl.w_o, d, P(L.z), d, x, d, M, d, d, r, skp, L.skp_bytes, s))
      return rc;
    if (int rc = norm(P(L.z), wl.g_mlp)) return rc;
    if (int rc = dec_gemm(P(L.h), d, wl.w_gate_up, d, P(L.uv), D.fw, nullptr, 0, M, D.fw, d, 1.f, skp,
                          L.skp_bytes, s))
      return rc;
    EltArgs a{};
    a.a = P(L.uv);
    a.out = P(L.s);
    a.rc = {nullptr, 1, M};
    a.f = static_cast<int32_t>(D.f);
    e = D.kind == LD_BLOCK_SWIGLU ? launch_swiglu_fwd(LD_BF16, a, s) : launch_relu2_fwd(LD_BF16, a, s);
    if (e != hipSuccess) return fail(LD_E_HIP, "activation: %s", hipGetErrorString(e));
    // x = z + r (s W_down^T)
    if (int rc = dec_gemm(P(L.s), D.f, wl.w_down, D.f, x, d, P(L.z), d, M, d, D.f, r, skp, L.skp_bytes, s))
      return rc;
  }
  return LD_OK;
}

// ------------------------------------------------------ kernel-level calls

int ld_rmsnorm_fwd(int32_t dtype, int32_t rows, int32_t d, float eps, const void* x, const void* g,
                   void* y, float* rstd, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || d < 1) return fail(LD_E_SHAPE, "bad shape");
  if (d % (dtype == LD_BF16 ? 8 : 4) || d > (dtype == LD_BF16 ? 4096 : 2048)) return fail(LD_E_SHAPE, "unsupported d");
  if (!(eps > 0.f)) return fail(LD_E_INVALID, "eps must be > 0");
  if (rows == 0) return LD_OK;
  if (!x || !g || !y || !rstd) return fail(LD_E_INVALID, "NULL pointer");
  RmsFwdArgs a{};
  a.x = x;
  a.src = {nullptr, 1};
  a.g = g;
  a.y = y;
  a.rstd = rstd;
  a.rc = {nullptr, 1, rows};
  a.d = d;
  a.eps = eps;
  hipError_t e = launch_rmsnorm_fwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "rmsnorm_fwd: %s", hipGetErrorString(e));
  return LD_OK;
}

size_t ld_rmsnorm_bwd_ws_bytes(int32_t rows, int32_t d) {
  if (rows < 0 || d < 1) return 0;
  return 4ull * rmsnorm_bwd_blocks(rows) * d;
}

int ld_rmsnorm_bwd(int32_t dtype, int32_t rows, int32_t d, const void* x, const void* g,
                   const float* rstd, const void* gy, const void* gres, void* gx, float* dg,
                   void* ws, size_t ws_bytes, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || d < 1) return fail(LD_E_SHAPE, "bad shape");
  if (d % (dtype == LD_BF16 ? 8 : 4) || d > (dtype == LD_BF16 ? 4096 : 2048)) return fail(LD_E_SHAPE, "unsupported d");
  if (!g || !dg || !ws || (rows > 0 && (!x || !rstd || !gy || !gx))) return fail(LD_E_INVALID, "NULL pointer");
  if (ws_bytes < ld_rmsnorm_bwd_ws_bytes(rows, d)) return fail(LD_E_WORKSPACE, "workspace too small");
  RmsBwdArgs a{};
  a.x = x;
  a.g = g;
  a.rstd = rstd;
  a.gy = gy;
  a.gres = gres;
  a.gx = gx;
  a.dst = {nullptr, 1};
  a.dg_part = static_cast<float*>(ws);
  a.rc = {nullptr, 1, rows};
  a.d = d;
  hipError_t e = launch_rmsnorm_bwd(dtype, a, dg, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "rmsnorm_bwd: %s", hipGetErrorString(e));
  return LD_OK;
}

int ld_swiglu_fwd(int32_t dtype, int32_t rows, int32_t f, const void* uv, void* s, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || f < 1 || f % (dtype == LD_BF16 ? 8 : 4)) return fail(LD_E_SHAPE, "bad shape");
  if (rows == 0) return LD_OK;
  if (!uv || !s) return fail(LD_E_INVALID, "NULL pointer");
  EltArgs a{};
  a.a = uv;
  a.out = s;
  a.rc = {nullptr, 1, rows};
  a.f = f;
  hipError_t e = launch_swiglu_fwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "swiglu_fwd: %s", hipGetErrorString(e));
  return LD_OK;
}

int ld_swiglu_bwd(int32_t dtype, int32_t rows, int32_t f, const void* uv, const void* gs,
                  void* guv, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || f < 1 || f % (dtype == LD_BF16 ? 8 : 4)) return fail(LD_E_SHAPE, "bad shape");
  if (rows == 0) return LD_OK;
  if (!uv || !gs || !guv) return fail(LD_E_INVALID, "NULL pointer");
  EltArgs a{};
  a.a = uv;
  a.b = gs;
  a.out = guv;
  a.rc = {nullptr, 1, rows};
  a.f = f;
  hipError_t e = launch_swiglu_bwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "swiglu_bwd: %s", hipGetErrorString(e));
  return LD_OK;
}

int ld_relu2_fwd(int32_t dtype, int32_t rows, int32_t f, const void* u, void* s, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || f < 1 || f % (dtype == LD_BF16 ? 8 : 4)) return fail(LD_E_SHAPE, "bad shape");
  if (rows == 0) return LD_OK;
  if (!u || !s) return fail(LD_E_INVALID, "NULL pointer");
  EltArgs a{};
  a.a = u;
  a.out = s;
  a.rc = {nullptr, 1, rows};
  a.f = f;
  hipError_t e = launch_relu2_fwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "relu2_fwd: %s", hipGetErrorString(e));
  return LD_OK;
}

int ld_relu2_bwd(int32_t dtype, int32_t rows, int32_t f, const void* u, const void* gs, void* gu,
                 void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (rows < 0 || f < 1 || f % (dtype == LD_BF16 ? 8 : 4)) return fail(LD_E_SHAPE, "bad shape");
  if (rows == 0) return LD_OK;
  if (!u || !gs || !gu) return fail(LD_E_INVALID, "NULL pointer");
  EltArgs a{};
  a.a = u;
  a.b = gs;
  a.out = gu;
  a.rc = {nullptr, 1, rows};
  a.f = f;
  hipError_t e = launch_relu2_bwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "relu2_bwd: %s", hipGetErrorString(e));
  return LD_OK;
}

float ld_alibi_slope(int32_t h, int32_t n_heads) { return alibi_slope(h, n_heads); }

size_t ld_gemm_skinny_ws_bytes(int32_t M, int32_t N, int32_t K) {
  if (M < 1 || M > kSkinnyMaxM || N < 1 || K < 0) return 0;
  return skinny_part_bytes(M, N, K);
}

int ld_gemm_skinny(int32_t M, int32_t N, int32_t K, const void* A, int32_t lda, const void* W, int32_t ldw,
                   void* C, int32_t ldc, float alpha, const void* R, int32_t ldr, void* ws, size_t ws_bytes,
                   void* stream) {
  t_err.clear();
  if (M < 1 || M > kSkinnyMaxM) return fail(LD_E_SHAPE, "M outside [1, %d]", kSkinnyMaxM);
  if (N < 1 || K < 0 || K % 8) return fail(LD_E_SHAPE, "need N >= 1, K >= 0, K %% 8 == 0");
  if (lda < K || ldw < K || ldc < N || (R && ldr < N)) return fail(LD_E_SHAPE, "leading dimension too small");
  if (lda % 8 || ldw % 8) return fail(LD_E_SHAPE, "lda, ldw must be multiples of 8");
  if (!A || !W || !C) return fail(LD_E_INVALID, "NULL pointer");
  if ((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(W)) & 15)
    return fail(LD_E_INVALID, "A and W must be 16-byte aligned");
  if (!std::isfinite(alpha)) return fail(LD_E_INVALID, "alpha not finite");
  const size_t need = ld_gemm_skinny_ws_bytes(M, N, K);
  if (need && (!ws || ws_bytes < need)) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  return dec_gemm(A, lda, W, ldw, C, ldc, R, ldr, M, N, K, alpha, static_cast<float*>(ws), ws ? ws_bytes : 0,
                  as_stream(stream));
}

int ld_gemm_dec(int32_t M, int32_t N, int32_t K, const void* A, int32_t lda, const void* g, float eps,
                const void* W, int32_t ldw, void* C, int32_t ldc, float alpha, const void* R, int32_t ldr,
                int32_t act, void* stream) {
  t_err.clear();
  if (M < 1 || M > kDecGemmMaxM) return fail(LD_E_SHAPE, "M outside [1, %d]", kDecGemmMaxM);
  if (N < 1 || K < 8 || K % 8) return fail(LD_E_SHAPE, "need N >= 1, K >= 8, K %% 8 == 0");
  if (act != kDecActNone && act != kDecActSwiglu && act != kDecActRelu2) return fail(LD_E_INVALID, "unknown act");
  if (act != kDecActNone && R) return fail(LD_E_INVALID, "a residual only without activation");
  if (!dec_gemm_ok(M, K, g != nullptr)) return fail(LD_E_UNSUPPORTED, "K = %d does not fit the staged rows", K);
  if (lda < K || ldw < K || ldc < N || (R && ldr < N)) return fail(LD_E_SHAPE, "leading dimension too small");
  if (lda % 8 || ldw % 8) return fail(LD_E_SHAPE, "lda, ldw must be multiples of 8");
  if (!A || !W || !C) return fail(LD_E_INVALID, "NULL pointer");
  if ((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(g)) & 15)
    return fail(LD_E_INVALID, "A, W and g must be 16-byte aligned");
  if (!std::isfinite(alpha)) return fail(LD_E_INVALID, "alpha not finite");
  if (g && !(eps > 0.f)) return fail(LD_E_INVALID, "eps must be > 0");
  return dec_proj(A, lda, g, eps, W, ldw, C, ldc, R, ldr, M, N, K, alpha, act, as_stream(stream));
}

int ld_kv_store(int32_t n_seq, int32_t n_new, int32_t d_model, int32_t pos, const void* qkv, void* kv,
                int32_t s_max, void* stream) {
  t_err.clear();
  if (n_seq < 1 || n_new < 1 || d_model < 8 || d_model % 8) return fail(LD_E_SHAPE, "bad sizes");
  if (pos < 0 || static_cast<int64_t>(pos) + n_new > s_max) return fail(LD_E_SHAPE, "positions outside the cache");
  if (!qkv || !kv) return fail(LD_E_INVALID, "NULL pointer");
  if ((reinterpret_cast<uintptr_t>(qkv) | reinterpret_cast<uintptr_t>(kv)) & 15)
    return fail(LD_E_INVALID, "qkv and kv must be 16-byte aligned");
  KvArgs k{};
  k.qkv = qkv;
  k.ld_qkv = 3ll * d_model;
  k.cache = kv;
  k.s_max = s_max;
  k.d = d_model;
  k.n = n_new;
  k.n_seq = n_seq;
  k.pos = pos;
  hipError_t e = launch_kv_store(k, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "kv store: %s", hipGetErrorString(e));
  return LD_OK;
}

size_t ld_attn_decode_ws_bytes(int32_t n_seq, int32_t n_heads, int32_t d_head, int32_t s_max) {
  if (n_seq < 1 || n_heads < 1 || d_head < 1 || s_max < 1) return 0;
  const size_t pc = static_cast<size_t>(n_seq) * n_heads * dec_chunks(s_max) * kDecMaxRows;
  return up(4 * pc * d_head) + up(4 * pc * 2);
}

int ld_attn_decode(int32_t n_seq, int32_t n_heads, int32_t d_head, int32_t alibi, int32_t pos, int32_t n_new,
                   const void* qkv, const void* kv, int32_t s_max, void* o, void* ws, size_t ws_bytes,
                   void* stream) {
  t_err.clear();
  if (d_head != 64 && d_head != 128) return fail(LD_E_UNSUPPORTED, "d_head must be 64 or 128");
  if (n_seq < 1 || n_heads < 1) return fail(LD_E_SHAPE, "n_seq, n_heads must be >= 1");
  if (n_new < 1 || n_new > kDecMaxRows) return fail(LD_E_INVALID, "n_new outside [1, %d]", kDecMaxRows);
  if (pos < 0 || static_cast<int64_t>(pos) + n_new > s_max) return fail(LD_E_SHAPE, "positions outside the cache");
  if (alibi != 0 && alibi != 1) return fail(LD_E_INVALID, "alibi must be 0 or 1");
  if (!qkv || !kv || !o || !ws) return fail(LD_E_INVALID, "NULL pointer");
  if ((reinterpret_cast<uintptr_t>(qkv) | reinterpret_cast<uintptr_t>(kv)) & 15)
    return fail(LD_E_INVALID, "qkv and kv must be 16-byte aligned");
  const size_t need = ld_attn_decode_ws_bytes(n_seq, n_heads, d_head, s_max);
  if (ws_bytes < need) return fail(LD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  const size_t pc = static_cast<size_t>(n_seq) * n_heads * dec_chunks(s_max) * kDecMaxRows;
  DecAttnArgs at{};
  at.qkv = qkv;
  at.ld_qkv = 3ll * n_heads * d_head;
  at.cache = kv;
  at.s_max = s_max;
  at.out = o;
  at.part_o = static_cast<float*>(ws);
  at.part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + up(4 * pc * d_head));
  at.n_seq = n_seq;
  at.H = n_heads;
  at.dh = d_head;
  at.n_new = n_new;
  at.pos = pos;
  at.n_chunks = static_cast<int32_t>(dec_chunks(static_cast<int64_t>(pos) + n_new));
  at.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(d_head)));
  at.alibi = alibi;
  hipError_t e = launch_attn_decode(at, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "attn decode: %s", hipGetErrorString(e));
  return LD_OK;
}

size_t ld_gemm_ws_bytes(int32_t dtype, int32_t a_kcontig, int32_t b_kcontig, int32_t M, int32_t N,
                        int32_t K, int32_t ldc, int32_t c_f32) {
  if (M < 1 || N < 1 || K < 0) return 0;
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.M = M;
  g.N = N;
  g.K = K;
  g.ldc = ldc;
  g.c_f32 = c_f32;
  const GemmPlan p = plan_gemm(dtype, a_kcontig ? 1 : 0, b_kcontig ? 1 : 0, g, M, K, true);
  return gemm_part_bytes(p, M, N);
}

int ld_gemm(int32_t dtype, int32_t a_kcontig, int32_t b_kcontig, int32_t M, int32_t N, int32_t K,
            const void* A, int32_t lda, const void* B, int32_t ldb, void* C, int32_t ldc,
            int32_t c_f32, float alpha, const void* R, int32_t ldr, void* ws, size_t ws_bytes,
            void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (M < 0 || N < 0 || K < 0) return fail(LD_E_SHAPE, "negative extent");
  if (M == 0 || N == 0) return LD_OK;
  if (!C || (K > 0 && (!A || !B))) return fail(LD_E_INVALID, "NULL pointer");
  if (dtype == LD_F32) c_f32 = 1;
  if (c_f32 && R && dtype == LD_BF16) return fail(LD_E_UNSUPPORTED, "float32 C with a residual needs LD_F32");
  if (ldc < N || (R && ldr < N)) return fail(LD_E_SHAPE, "ldc/ldr smaller than N");
  if (K > 0) {
    if (lda < (a_kcontig ? K : M) || ldb < (b_kcontig ? K : N)) return fail(LD_E_SHAPE, "lda/ldb too small");
    if (dtype == LD_BF16) {
      if (lda % 8 || ldb % 8) return fail(LD_E_SHAPE, "bf16 needs lda, ldb multiples of 8");
      if ((a_kcontig || b_kcontig) && K % 8) return fail(LD_E_SHAPE, "bf16 needs K %% 8 == 0");
      if ((!a_kcontig && M % 8) || (!b_kcontig && N % 8))
        return fail(LD_E_SHAPE, "bf16 needs M (N) %% 8 == 0 for a k-strided A (B)");
    }
  }
  GemmArgs g = gemm_args();
  g.A = A;
  g.B = B;
  g.C = C;
  g.R = R;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.ldr = ldr;
  g.M = M;
  g.N = N;
  g.K = K;
  g.out_map = {nullptr, 1};
  g.alpha = alpha;
  g.c_f32 = c_f32;
  return run_gemm(dtype, a_kcontig ? 1 : 0, b_kcontig ? 1 : 0, g, M, M, K, as_stream(stream),
                  static_cast<float*>(ws), ws ? ws_bytes : 0, K);
}

int ld_attn_fwd(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                int32_t alibi, const void* qkv, void* o, float* lse, void* stream) {
  t_err.clear();
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (n_seq < 0 || seq < 1 || n_heads < 1) return fail(LD_E_SHAPE, "bad shape");
  if (dtype == LD_BF16 ? (d_head != 64 && d_head != 128) || seq % 64
                       : (d_head != 16 && d_head != 32 && d_head != 64))
    return fail(LD_E_UNSUPPORTED, "unsupported d_head/seq");
  if (alibi != 0 && alibi != 1) return fail(LD_E_INVALID, "alibi must be 0 or 1");
  if (n_seq == 0) return LD_OK;
  if (!qkv || !o || !lse) return fail(LD_E_INVALID, "NULL pointer");
  AttnArgs a{};
  a.qkv = qkv;
  a.out = o;
  a.lse = lse;
  a.n_seq = n_seq;
  a.S = seq;
  a.H = n_heads;
  a.dh = d_head;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(d_head)));
  a.alibi = alibi;
  hipError_t e = launch_attn_fwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "attn_fwd: %s", hipGetErrorString(e));
  return LD_OK;
}

size_t ld_attn_bwd_ws_bytes(int32_t n_seq, int32_t seq, int32_t n_heads) {
  if (n_seq < 0 || seq < 1 || n_heads < 1) return 0;
  return 4ull * n_seq * seq * n_heads;
}

namespace {
int attn_bwd_common(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head, int32_t alibi,
                    const void* qkv, const void* o, const float* lse, const void* go, void* gqkv, float* delta,
                    void* stream) {
  AttnArgs a{};
  a.qkv = qkv;
  a.o = o;
  a.go = go;
  a.out = gqkv;
  a.lse = const_cast<float*>(lse);
  a.delta = delta;
  a.n_seq = n_seq;
  a.S = seq;
  a.H = n_heads;
  a.dh = d_head;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(d_head)));
  a.alibi = alibi;
  hipError_t e = launch_attn_bwd(dtype, a, as_stream(stream));
  if (e != hipSuccess) return fail(LD_E_HIP, "attn_bwd: %s", hipGetErrorString(e));
  return LD_OK;
}

int check_attn_bwd(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head, int32_t alibi) {
  if (dtype != LD_F32 && dtype != LD_BF16) return fail(LD_E_INVALID, "unknown dtype");
  if (n_seq < 0 || seq < 1 || n_heads < 1) return fail(LD_E_SHAPE, "bad shape");
  if (dtype == LD_BF16 ? (d_head != 64 && d_head != 128) || seq % 64
                       : (d_head != 16 && d_head != 32 && d_head != 64))
    return fail(LD_E_UNSUPPORTED, "unsupported d_head/seq");
  if (alibi != 0 && alibi != 1) return fail(LD_E_INVALID, "alibi must be 0 or 1");
  return LD_OK;
}
}  // namespace

int ld_attn_bwd(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                int32_t alibi, const void* qkv, const void* o, const float* lse, const void* go,
                void* gqkv, void* ws, size_t ws_bytes, void* stream) {
  t_err.clear();
  if (int rc = check_attn_bwd(dtype, n_seq, seq, n_heads, d_head, alibi)) return rc;
  if (n_seq == 0) return LD_OK;
  if (!qkv || !o || !lse || !go || !gqkv || !ws) return fail(LD_E_INVALID, "NULL pointer");
  if (ws_bytes < ld_attn_bwd_ws_bytes(n_seq, seq, n_heads)) return fail(LD_E_WORKSPACE, "workspace too small");
  return attn_bwd_common(dtype, n_seq, seq, n_heads, d_head, alibi, qkv, o, lse, go, gqkv,
                         static_cast<float*>(ws), stream);
}

int ld_attn_bwd_noalloc(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                        int32_t alibi, const void* qkv, const void* o, const float* lse, const void* go,
                        void* gqkv, void* stream) {
  t_err.clear();
  if (int rc = check_attn_bwd(dtype, n_seq, seq, n_heads, d_head, alibi)) return rc;
  if (n_seq == 0) return LD_OK;
  if (!qkv || !o || !lse || !go || !gqkv) return fail(LD_E_INVALID, "NULL pointer");
  const size_t need = ld_attn_bwd_ws_bytes(n_seq, seq, n_heads);
  if (need > kAttnScratchBytes)
    return fail(LD_E_UNSUPPORTED, "n_seq * n_heads * seq = %lld exceeds the fixed scratch (%zu bytes, %zu rows)",
                static_cast<long long>(need / 4), kAttnScratchBytes, kAttnScratchBytes / 4);
  float* delta = nullptr;
  hipError_t e = attn_scratch_ptr(&delta);
  if (e != hipSuccess) return fail(LD_E_HIP, "scratch address: %s", hipGetErrorString(e));
  return attn_bwd_common(dtype, n_seq, seq, n_heads, d_head, alibi, qkv, o, lse, go, gqkv, delta, stream);
}

// -------------------------------------------------------------- profiling

int ld_prof_start(const char* kernel_name) {
  t_err.clear();
  if (!kernel_name) return fail(LD_E_INVALID, "kernel_name is NULL");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.name = kernel_name;
  g_prof.recs.clear();
  g_prof.next = 0;
  g_prof.on = true;
  return LD_OK;
}

int ld_prof_stop(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  return LD_OK;
}

int ld_prof_result(int64_t* launches, double* total_ms, double* flops, double* bytes) {
  t_err.clear();
  if (!launches || !total_ms || !flops || !bytes) return fail(LD_E_INVALID, "NULL pointer");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  double ms = 0, fl = 0, by = 0;
  for (const ProfRec& r : g_prof.recs) {
    LD_HIP(hipEventSynchronize(r.e1));
    float t = 0.f;
    LD_HIP(hipEventElapsedTime(&t, r.e0, r.e1));
    ms += t;
    fl += r.flops;
    by += r.bytes;
  }
  *launches = static_cast<int64_t>(g_prof.recs.size());
  *total_ms = ms;
  *flops = fl;
  *bytes = by;
  return LD_OK;
}

}  // extern "C"

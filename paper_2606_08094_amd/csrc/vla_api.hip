// Host runtime of libvla: argument validation, model creation (weights copied
// and re-tiled into library-owned memory), the launch plan of one denoising
// integration, its capture into a HIP graph, and the C ABI entry points.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
#include <memory>
#include <string>
#include <tuple>
#include <vector>

#include "vla.h"
#include "vla_internal.h"
#include "vla_test.h"

namespace {

thread_local std::string g_err;

vla_status fail(vla_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(VLA_E_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define VLA_TRY(expr)                 \
  do {                                \
    vla_status s_ = (expr);           \
    if (s_ != VLA_OK) return s_;      \
  } while (0)

inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

enum Kind { K_SELF = 0, K_CROSS = 1, K_JOINT = 2, K_MLP = 3 };

std::vector<int> sublayers(const vla_config& c, int l) {
  switch (c.pattern) {
    case VLA_PAT_SELF_CROSS: return {K_SELF, K_CROSS, K_MLP};
    case VLA_PAT_JOINT: return {K_JOINT, K_MLP};
    case VLA_PAT_CROSS: return {K_CROSS, K_MLP};
    default: return (l % 2 == 0) ? std::vector<int>{K_CROSS, K_MLP} : std::vector<int>{K_SELF, K_MLP};
  }
}
int n_sub(const vla_config& c) { return c.pattern == VLA_PAT_SELF_CROSS ? 3 : 2; }
bool has_prefix(int kind) { return kind == K_CROSS || kind == K_JOINT; }
bool has_self(int kind) { return kind == K_SELF || kind == K_JOINT; }

int cache_layers(const vla_config& c) {
  int n = 0;
  for (int l = 0; l < c.n_layers; ++l)
    for (int k : sublayers(c, l)) n += has_prefix(k) ? 1 : 0;
  return n;
}

vla_status validate_config(const vla_config* c) {
  if (!c) return fail(VLA_E_ARG, "config is NULL");
  if (c->pattern < 0 || c->pattern > 3) return fail(VLA_E_ARG, "pattern %d out of range", c->pattern);
  if (c->mlp < 0 || c->mlp > 3) return fail(VLA_E_ARG, "mlp %d out of range", c->mlp);
  if (c->wtype < 0 || c->wtype > 2) return fail(VLA_E_ARG, "wtype %d out of range", c->wtype);
  if (c->n_layers < 1 || c->d_model < 2 || c->n_heads < 1 || c->n_kv_heads < 1 || c->d_ff < 16 ||
      c->d_prefix < 1 || c->n_action < 1 || c->d_action < 1 || c->d_state < 0)
    return fail(VLA_E_SHAPE, "non-positive dimension in config");
  if (c->d_model % 2) return fail(VLA_E_SHAPE, "d_model must be even (sinusoidal time embedding)");
  if (c->n_heads % c->n_kv_heads) return fail(VLA_E_SHAPE, "n_heads %% n_kv_heads != 0");
  const bool f32 = c->wtype == VLA_W_F32;
  if (f32 ? !(c->head_dim == 64 || c->head_dim == 128) : !(c->head_dim == 64 || c->head_dim == 128 || c->head_dim == 256))
    return fail(VLA_E_UNSUPPORTED, "head_dim %d unsupported (64, 128%s)", c->head_dim, f32 ? "" : ", 256");
  const int vk = f32 ? 4 : 8;
  if (c->d_model % vk || c->d_prefix % vk || (c->n_heads * c->head_dim) % vk || c->d_ff % 16)
    return fail(VLA_E_SHAPE, "d_model, d_prefix, H*hd must be multiples of %d and d_ff of 16", vk);
  if (c->wtype == VLA_W_TERNARY) {
    if (c->d_model % 64 || c->d_prefix % 64 || (c->n_heads * c->head_dim) % 64 || c->d_ff % 64)
      return fail(VLA_E_SHAPE, "ternary weights need every K (d, d_p, H*hd, F) to be a multiple of 64");
  }
  if (c->d_action > 64) return fail(VLA_E_UNSUPPORTED, "d_action > 64");
  if (c->n_heads / c->n_kv_heads > 8 || c->n_heads > 32)
    return fail(VLA_E_UNSUPPORTED, "more than 8 query heads per K/V head or more than 32 heads");
  if (c->head_regression != 0 && c->head_regression != 1) return fail(VLA_E_ARG, "head_regression must be 0/1");
  if (!(c->rms_eps > 0.0f) || !std::isfinite(c->rms_eps)) return fail(VLA_E_ARG, "rms_eps must be finite and > 0");
  if (c->n_action > 4096 || c->d_model > 16384 || c->d_ff > 65536)
    return fail(VLA_E_UNSUPPORTED, "dimension beyond the supported range");
  return VLA_OK;
}

// ----------------------------------------------------------------------------
// Model

struct SubW {
  int kind = K_MLP;
  int cache_idx = -1;
  // dense (element type)
  void* qkv = nullptr;  // [n_qkv][d]: W_q | W_k | W_v (self/joint) or W_q (cross)
  int n_qkv = 0;
  void* kvc = nullptr;  // [2 d_kv][d_p]: W_kc | W_vc
  void* o = nullptr;    // [d][d_q]
  void* gu = nullptr;   // GLU: [2F][d] gate/up interleaved in 16-row blocks; GELU: W1 [F][d]
  void* dn = nullptr;   // [d][F]
  // ternary: same matrices packed [N][K/4], per-row scale vectors
  float *s_qkv = nullptr, *s_kvc = nullptr, *s_o = nullptr, *s_gu = nullptr, *s_dn = nullptr;
};

struct Plan;
struct PrefixWs;

}  // namespace

struct vla_model {
  vla_config cfg{};
  int et = ET_BF16;     // element type of dense matrices and activations
  bool tern = false;
  int d = 0, dq = 0, dkv = 0, ns = 0, Lc = 0;
  std::vector<void*> allocs;
  void *W_in = nullptr, *W_s = nullptr, *E_pos = nullptr, *W_out = nullptr;
  void* kvc_all = nullptr;  // dense models: every cache slot's [W_kc | W_vc] stacked in slot order
  float *b_in = nullptr, *b_s = nullptr, *b_out = nullptr;
  void *W_t1 = nullptr, *W_t2 = nullptr, *W_fm = nullptr, *W_mod = nullptr;
  float *b_t1 = nullptr, *b_t2 = nullptr, *b_fm = nullptr, *b_mod = nullptr;
  float *mod_static = nullptr, *modf_static = nullptr;
  std::vector<std::vector<SubW>> layers;
  // persistent kernel: each layer's W_d (or W2) once more, team-major (team t's
  // d_ff / 8 columns as one [d][d_ff / 8] block); built on the first persistent plan
  std::vector<const void*> wd_team;
  std::map<std::tuple<int, int, int, int>, std::unique_ptr<Plan>> plans;
  std::map<std::pair<int, int>, std::unique_ptr<PrefixWs>> prefix_ws;
  int loop_mode = 2;
  int profile = 0;
  int trace = 0;                  // record the persistent kernel's phase timeline
  int causal = 0;                 // causal action-token attention (VLA_OPT_CAUSAL_SELF)
  int state_token = 0;            // state as its own leading token (VLA_OPT_STATE_TOKEN)
  float rope_base = 0.0f;         // rotary position embedding base, 0 = none (VLA_OPT_ROPE_BASE)
  int attn_splits = 0;            // key splits of the launch-per-phase attention (0 = automatic)
  long spin_limit = PERSIST_SPIN_DEFAULT;  // persistent kernel: polls of a barrier wait (VLA_OPT_PERSIST_SPIN_LIMIT)
  int persist_dev_ok = -1;        // the device holds the persistent kernel's whole grid (-1 = not yet asked)
  void* last_profiled = nullptr;  // Plan* of the last profiled call
  void* last_traced = nullptr;    // Plan* of the last traced call
  hipStream_t cap_stream = nullptr;
  ~vla_model();
};

namespace {

size_t esize(int et) { return et == ET_BF16 ? 2 : 4; }

struct Alloc {
  std::vector<void*>& list;
  vla_status operator()(void** p, size_t bytes) {
    *p = nullptr;
    if (bytes == 0) bytes = 16;
    if (hipMalloc(p, bytes) != hipSuccess) {
      *p = nullptr;
      return fail(VLA_E_NOMEM, "hipMalloc(%zu) failed", bytes);
    }
    list.push_back(*p);
    return VLA_OK;
  }
};

// Reads weight-table entries in order.
struct TableReader {
  const void* const* w;
  int n, i = 0;
  vla_status next(const void** p, const char* what) {
    if (i >= n) return fail(VLA_E_ARG, "weight table too short at %s", what);
    *p = w[i++];
    if (!*p) return fail(VLA_E_ARG, "weight %s (entry %d) is NULL", what, i - 1);
    if (!al16(*p)) return fail(VLA_E_ARG, "weight %s (entry %d) is not 16-byte aligned", what, i - 1);
    return VLA_OK;
  }
};

}  // namespace

// ----------------------------------------------------------------------------
// Plans: one denoising integration for (batch, prefix_len, n_steps).

namespace {

struct Op {
  std::function<hipError_t(hipStream_t)> fn;
  vla_op_time info;
  hipError_t operator()(hipStream_t s) const { return fn(s); }
};

vla_op_time op_info(int kind, int M, int N, int K, double bytes, double flops) {
  vla_op_time t{};
  t.kind = kind;
  t.M = M;
  t.N = N;
  t.K = K;
  t.bytes = bytes;
  t.flops = flops;
  return t;
}

struct Plan {
  int B = 0, P = 0, T = 0;
  bool persist = false;       // one launch of co-resident workgroups runs the whole step loop
  std::vector<void*> allocs;
  CallParams* cp = nullptr;
  float *a = nullptr, *xs = nullptr, *x = nullptr, *mods = nullptr, *modf = nullptr;
  void* u = nullptr;          // adaRMS output, input of the next projection
  float* part = nullptr;      // split-K partials of the residual projections
  void *e = nullptr, *h1 = nullptr, *sc = nullptr, *qkv = nullptr, *o = nullptr, *h = nullptr;
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  void* apart = nullptr;      // attention key-split partials
  float* astats = nullptr;
  std::vector<Op> ops;
  hipGraphExec_t exec = nullptr;
  std::vector<hipEvent_t> events;  // 2 per op when profiled
  int prof_reps = 1;
  int* persist_err = nullptr;       // persistent kernel: set if a barrier timed out (device word)
  int* persist_err_host = nullptr;  // pinned host copy of it, written after every launch
  unsigned long long* trace = nullptr;  // persistent kernel: phase timeline (8 x PERSIST_TRACE_MAX)
  ~Plan() {
    if (persist_err_host) {
      (void)hipDeviceSynchronize();   // no copy into the host word is still in flight
      (void)hipHostFree(persist_err_host);
    }
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
    if (exec) (void)hipGraphExecDestroy(exec);
    for (void* p : allocs) (void)hipFree(p);
  }
};

struct PrefixWs {
  std::vector<void*> allocs;
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  ~PrefixWs() {
    for (void* p : allocs) (void)hipFree(p);
  }
};

struct Tiling {
  int ms, nsub, nc, nsplit, n_tiles, m_tiles, units;
};

// W2A8 GEMM: 64*nsub W rows per workgroup over the whole K (K-slices of
// 256*nc looped inside the workgroup).
Tiling tern_tiling(int M, int N, int K, int nsub) {
  Tiling t{};
  t.ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  t.nsub = nsub;
  t.m_tiles = cdiv(M, 16 * t.ms);
  t.n_tiles = cdiv(N, 64 * nsub);
  t.nc = K <= 256 ? 1 : K <= 512 ? 2 : K <= 1024 ? 4 : 8;
  t.nsplit = 1;
  t.units = t.m_tiles * t.n_tiles;
  return t;
}

// Dense GEMM launch: the skinny kernel when the shape allows (M <= 128), else
// the tiled one (bf16) or the wide one (fp32).
struct DenseLaunch {
  bool skinny;
  bool tile;
  SkinnyShape sk;
  WideShape wd;
  TileShape tl;
  // K-splits whose fp32 partials a later kernel sums (EPI_PARTIAL only)
  int splits() const { return skinny ? sk.nsplit : (tile ? tl.nsplit : 1); }
};

// variant: 0 = the runtime's choice (split-K only for EPI_PARTIAL), 1 = wide,
// 2 = skinny, 3 = tiled, 10 + i = tiled with tile i fixed.
DenseLaunch dense_launch(int et, const GemmArgs& a, int nsub, int variant = 0) {
  DenseLaunch d{};
  const bool split_ok = a.epi == EPI_PARTIAL;
  if (variant == 0 || variant == 2) d.skinny = skinny_plan(et, a.M, a.N, a.K, nsub, split_ok, &d.sk);
  if (!d.skinny && (variant == 0 || variant == 3 || variant >= 10))
    d.tile = tile_plan(et, a.M, a.N, a.K, split_ok, variant >= 10 ? variant - 10 : -1, &d.tl);
  if (!d.skinny && !d.tile) wide_plan(et, a.M, a.N, a.K, nsub, &d.wd);
  return d;
}

hipError_t launch_dense(int et, const DenseLaunch& d, const GemmArgs& a, hipStream_t s) {
  if (d.skinny) return launch_gemm_skinny(et, d.sk, a, s);
  if (d.tile) return launch_gemm_tile(d.tl, a, s);
  return launch_gemm_wide(et, d.wd, a, s);
}

// Collects the launches of a plan and the workspace they need.
struct Builder {
  vla_model* m;
  std::vector<Op>* ops;
  void** apart;
  float** astats;
  size_t part_need = 0, stats_need = 0;

  void gemm(GemmArgs a, int nsub) {
    const int et = m->et;
    const DenseLaunch dl = dense_launch(et, a, nsub);
    const double es = esize(et);
    const double xb = es;
    double ob = a.out_f32 ? 4.0 : es;
    // split-K partials are this implementation's traffic, not the method's:
    // the projection's output counts once, as one fp32 array
    if (a.epi == EPI_PARTIAL) ob = 4.0;
    if (a.epi == EPI_RESID) ob = 8.0;                           // residual read + write
    if (a.epi == EPI_GLU) ob = es * 0.5;                        // one output per gate/up pair
    const double bytes = (double)a.N * a.K * es + (double)a.M * a.K * xb + (double)a.M * a.N * ob;
    ops->push_back(Op{[=](hipStream_t s) { return launch_dense(et, dl, a, s); },
                      op_info(nsub == 2 ? VLA_OP_GEMM_GLU : VLA_OP_GEMM, a.M, a.N, a.K, bytes,
                              2.0 * a.M * a.N * a.K)});
  }

  void tern(TernArgs a, int nsub) {
    const Tiling t = tern_tiling(a.M, a.N, a.K, nsub);
    a.ks = t.nc * 256;
    a.nsplit = 1;
    a.n_tiles = t.n_tiles;
    double ob = a.e.out_f32 ? 4.0 : 2.0;
    if (a.e.epi == EPI_RESID) ob = 8.0;
    if (a.e.epi == EPI_GLU) ob = 2.0;
    const double bytes = (double)a.N * a.K / 4.0 + (double)a.M * a.K + (double)a.M * a.N * ob;
    ops->push_back(Op{[=](hipStream_t s) { return launch_ternary_gemm(a, t.ms, t.units, s); },
                      op_info(VLA_OP_TERNARY, a.M, a.N, a.K, bytes, 2.0 * a.M * a.N * a.K)});
  }

  void attn(AttnArgs a) {
    const int QT = cdiv(a.n, 16);
    const int total = (a.mode == 0 ? 0 : a.P) + (a.mode == 1 ? 0 : a.n);
    (void)QT;
    const int et = m->et;
    attention_split(a, m->attn_splits % 100, m->attn_splits / 100);
    if (m->attn_splits == 0 && attention_tile_eligible(et, a)) attention_tile_split(a, 0);
    part_need = std::max(part_need, attention_part_bytes(et, a));
    stats_need = std::max(stats_need, attention_stats_bytes(a));
    void** pp = apart;
    float** sp = astats;
    const double es = esize(et);
    const double keys = total;
    const double bytes = (double)a.B * a.G * (a.mode == 0 ? 0 : a.P) * a.hd * 2 * es +  // cached K/V
                         (double)a.B * a.n * (2.0 * a.H * a.hd + (a.mode == 1 ? 0 : 2.0 * a.G * a.hd)) * es;
    const bool split = a.kv_split > 1;
    // Key-split partials (element type) plus (m, l) per split: traffic of this
    // implementation, not of the method, so only the merge reports them.
    const double pbytes = split ? (double)a.kv_split * a.B * a.n * a.H * (a.hd * es + 8.0) : 0.0;
    ops->push_back(Op{[=](hipStream_t s) {
                        AttnArgs g = a;
                        g.part = *pp;
                        g.stats = *sp;
                        return launch_attention(et, g, s, 1);
                      },
                      op_info(VLA_OP_ATTENTION, a.B * a.n, (int)keys, a.hd, bytes,
                              4.0 * a.B * a.n * a.H * a.hd * keys)});
    if (split)
      ops->push_back(Op{[=](hipStream_t s) {
                          AttnArgs g = a;
                          g.part = *pp;
                          g.stats = *sp;
                          return launch_attention(et, g, s, 2);
                        },
                        op_info(VLA_OP_ATTN_MERGE, a.B * a.n, a.kv_split, a.hd,
                                pbytes + (double)a.B * a.n * a.H * a.hd * es, 0.0)});
  }

  void row_norm(RowNormArgs r) {
    const int et = m->et;
    const double es = esize(et);
    const double bytes = (double)r.M * r.d * (8.0 + 4.0 * std::min(r.nsplit, 1) + (r.u_f32 ? 4.0 : es)) +
                         (r.mode == 1 ? (double)r.d * (r.A + r.n) * es : 0.0);
    ops->push_back(Op{[=](hipStream_t s) { return launch_row_norm(et, r, s); },
                      op_info(VLA_OP_SMALL, r.M, r.d, r.nsplit, bytes, 0.0)});
  }

  void quant(QuantArgs q) {
    const double bytes = (double)q.M * q.K * ((q.src_type == 1 ? 2.0 : 4.0) + 1.0);
    ops->push_back(Op{[=](hipStream_t s) { return launch_quantize(q, s); },
                      op_info(VLA_OP_QUANTIZE, q.M, 0, q.K, bytes, 0.0)});
  }

  void small(std::function<hipError_t(hipStream_t)> f, int M, int N, int K, double bytes) {
    ops->push_back(Op{std::move(f), op_info(VLA_OP_SMALL, M, N, K, bytes, 0.0)});
  }
};

GemmArgs gemm_base(const vla_model* m, int M, int N, int K, const void* X, int ldx, const void* W) {
  GemmArgs a{};
  a.M = M;
  a.N = N;
  a.K = K;
  a.X = X;
  a.ldx = ldx;
  a.W = W;
  (void)m;
  return a;
}

int mlp_act(int mlp) {
  switch (mlp) {
    case VLA_MLP_GELU:
    case VLA_MLP_GEGLU: return ACT_GELU;
    case VLA_MLP_SWIGLU: return ACT_SILU;
    default: return ACT_RELU2;
  }
}

// The persistent step kernel covers the batch-1 bf16 dense expert with joint
// attention whose shape fits its team layout (see persist_supported).
bool persist_eligible(vla_model* m, int B, int P, int T) {
  // its attention is unmasked and unrotated, its rows are the action tokens alone
  if (m->causal || m->rope_base > 0.0f || m->state_token) return false;
  const vla_config& c = m->cfg;
  int kba = 0, nsplit = 0;
  const bool shape_ok = !m->tern && m->et == ET_BF16 && c.pattern == VLA_PAT_JOINT && !c.head_regression &&
                        B == 1 && T >= 1 && c.n_layers >= 1 && c.n_layers <= PERSIST_MAX_LAYERS &&
                        persist_supported(m->d, c.head_dim, c.n_heads, c.n_kv_heads, c.d_ff, c.n_action, P,
                                          c.d_action, c.mlp != VLA_MLP_GELU, &kba, &nsplit);
  if (!shape_ok) return false;
  if (m->persist_dev_ok < 0) m->persist_dev_ok = persist_resident(m->d, c.head_dim, c.n_heads / 8) ? 1 : 0;
  return m->persist_dev_ok == 1;
}

// A device-side failure of an earlier call (a persistent-kernel barrier that
// timed out) that has become visible on the host: report it once.
vla_status take_device_error(vla_model* m) {
  for (auto& kv : m->plans) {
    Plan* p = kv.second.get();
    if (p->persist_err_host && *reinterpret_cast<volatile int*>(p->persist_err_host) != 0) {
      *reinterpret_cast<volatile int*>(p->persist_err_host) = 0;
      return fail(VLA_E_DEVICE, "an earlier vla_denoise failed on the device: a barrier of the persistent "
                                "kernel timed out, and that call's actions_out holds NaN");
    }
  }
  return VLA_OK;
}

vla_status build_plan(vla_model* m, Plan* p) {
  const vla_config& c = m->cfg;
  const int B = p->B, P = p->P, T = p->T;
  const int n = c.n_action, A = c.d_action, S = c.d_state, d = m->d, F = c.d_ff;
  // token rows per request: the n action tokens, after the state token when it is on
  const int nt = n + (m->state_token ? 1 : 0), stok = m->state_token ? nt : 0;
  const int M = B * nt, L = c.n_layers, ns = m->ns, dq = m->dq, dkv = m->dkv, hd = c.head_dim;
  const int et = m->et;
  const size_t es = esize(et);
  const bool u32 = m->tern || et == ET_F32;   // W2A8 quantiser input and fp32 models keep u in fp32
  const size_t modrow = (size_t)L * 3 * ns * d;
  Alloc al{p->allocs};
  VLA_TRY(al((void**)&p->cp, sizeof(CallParams)));
  VLA_TRY(al((void**)&p->a, (size_t)B * n * A * 4));
  VLA_TRY(al((void**)&p->xs, (size_t)B * d * 4));
  VLA_TRY(al((void**)&p->x, (size_t)M * d * 4));
  VLA_TRY(al(&p->u, (size_t)M * d * (u32 ? 4 : es)));
  int ldqkv = 0;
  for (auto& lay : m->layers)
    for (auto& sw : lay) ldqkv = std::max(ldqkv, sw.n_qkv);
  VLA_TRY(al(&p->qkv, (size_t)M * ldqkv * es));
  VLA_TRY(al(&p->o, (size_t)M * dq * es));
  VLA_TRY(al(&p->h, (size_t)M * F * (m->tern ? 4 : es)));
  if (!c.head_regression) {
    VLA_TRY(al(&p->e, (size_t)T * d * es));
    VLA_TRY(al(&p->h1, (size_t)T * d * es));
    VLA_TRY(al(&p->sc, (size_t)T * d * es));
    VLA_TRY(al((void**)&p->mods, (size_t)T * modrow * 4));
    VLA_TRY(al((void**)&p->modf, (size_t)T * 2 * d * 4));
  }
  if (m->tern) {
    VLA_TRY(al((void**)&p->q8, (size_t)M * std::max(std::max(d, dq), F)));
    VLA_TRY(al((void**)&p->r8, (size_t)M * 4));
  }

  Builder bld{m, &p->ops, &p->apart, &p->astats};
  CallParams* cp = p->cp;
  size_t part_need = 0;

  // chunk start and (flow heads) the time embedding of every solver step, one launch;
  // with the state token b_in belongs to the action rows only, added by the embedding
  void* temb = c.head_regression ? nullptr : p->e;
  bld.small([=](hipStream_t s) {
    return launch_chunk_start(et, cp, p->a, p->xs, m->W_s, m->b_s, stok ? nullptr : m->b_in, B, n, A, S, d,
                              temb, T, T, s);
  }, B, d, S, (double)d * S * es + (double)B * (S + d) * 4 + (double)B * n * A * 8 + (temb ? (double)T * d * es : 0.0));
  if (!c.head_regression) {
    GemmArgs g = gemm_base(m, T, d, d, p->e, d, m->W_t1);
    g.epi = EPI_STORE;
    g.bias = m->b_t1;
    g.act = ACT_SILU;
    g.out = p->h1;
    g.ldo = d;
    bld.gemm(g, 1);
    g = gemm_base(m, T, d, d, p->h1, d, m->W_t2);
    g.epi = EPI_STORE;
    g.bias = m->b_t2;
    g.act = ACT_SILU;
    g.out = p->sc;
    g.ldo = d;
    bld.gemm(g, 1);
    g = gemm_base(m, T, (int)modrow, d, p->sc, d, m->W_mod);
    g.epi = EPI_STORE;
    g.bias = m->b_mod;
    g.out = p->mods;
    g.ldo = (int)modrow;
    g.out_f32 = 1;
    bld.gemm(g, 1);
    g = gemm_base(m, T, 2 * d, d, p->sc, d, m->W_fm);
    g.epi = EPI_STORE;
    g.bias = m->b_fm;
    g.out = p->modf;
    g.ldo = 2 * d;
    g.out_f32 = 1;
    bld.gemm(g, 1);
  }

  if (p->persist) {
    PersistArgs pa{};
    pa.L = L; pa.d = d; pa.H = c.n_heads; pa.G = c.n_kv_heads; pa.hd = hd; pa.F = F; pa.n = n; pa.P = P;
    pa.A = A; pa.T = T;
    pa.glu = c.mlp != VLA_MLP_GELU;
    pa.act = mlp_act(c.mlp);
    pa.HT = c.n_heads / 8;
    if (!persist_supported(d, hd, c.n_heads, c.n_kv_heads, F, n, P, A, pa.glu, &pa.kba, &pa.nsplit))
      return fail(VLA_E_UNSUPPORTED, "persistent kernel: unsupported shape");
    pa.eps = c.rms_eps;
    pa.scale = 1.0f / std::sqrt((float)hd);
    const size_t layer_block = (size_t)2 * B * c.n_kv_heads * P * hd;
    // Team t reads only columns [t F / 8, (t + 1) F / 8) of W_d: one contiguous
    // block per team instead of d pieces of F / 4 bytes, F * es bytes apart.
    if (m->wd_team.empty()) {
      Alloc am{m->allocs};
      const size_t F8 = (size_t)F / 8;
      std::vector<const void*> wt(L);
      for (int l = 0; l < L; ++l) {
        void* dst = nullptr;
        VLA_TRY(am(&dst, (size_t)d * F * es));
        const char* src = static_cast<const char*>(m->layers[l][1].dn);
        for (int t = 0; t < 8; ++t)
          HIP_TRY(hipMemcpy2D(static_cast<char*>(dst) + t * d * F8 * es, F8 * es, src + t * F8 * es, (size_t)F * es,
                              F8 * es, d, hipMemcpyDeviceToDevice));
        wt[l] = dst;
      }
      HIP_TRY(hipDeviceSynchronize());
      m->wd_team = wt;
    }
    std::vector<PLayer> hl(L);
    for (int l = 0; l < L; ++l) {
      const std::vector<SubW>& subs = m->layers[l];
      if (subs.size() != 2 || subs[0].kind != K_JOINT || subs[1].kind != K_MLP)
        return fail(VLA_E_UNSUPPORTED, "persistent kernel: layer %d is not joint attention + MLP", l);
      hl[l].wqkv = subs[0].qkv;
      hl[l].wo = subs[0].o;
      hl[l].wgu = subs[1].gu;
      hl[l].wd = m->wd_team[l];
      hl[l].cache_off = (size_t)subs[0].cache_idx * layer_block;
    }
    PLayer* dl = nullptr;
    VLA_TRY(al((void**)&dl, sizeof(PLayer) * L));
    HIP_TRY(hipMemcpy(dl, hl.data(), sizeof(PLayer) * L, hipMemcpyHostToDevice));
    pa.layers = dl;
    pa.cp = cp;
    pa.mods = p->mods;
    pa.modf = p->modf;
    // W_in zero-padded to [d][32] so the kernel's embedding reads aligned,
    // fixed-length rows
    void* win_pad = nullptr;
    VLA_TRY(al(&win_pad, (size_t)d * 32 * 2));
    HIP_TRY(hipMemset(win_pad, 0, (size_t)d * 32 * 2));
    HIP_TRY(hipMemcpy2D(win_pad, 32 * 2, m->W_in, (size_t)A * 2, (size_t)A * 2, d, hipMemcpyDeviceToDevice));
    pa.w_in = win_pad;
    pa.xs = p->xs;
    pa.e_pos = m->E_pos;
    pa.w_out = m->W_out;
    pa.b_out = m->b_out;
    pa.a0 = p->a;
    const int HT = pa.HT;
    VLA_TRY(al(&pa.u, (size_t)8 * n * d * 2));
    VLA_TRY(al(&pa.qkv, (size_t)8 * n * (HT + 2) * hd * 2));
    VLA_TRY(al(&pa.apart, (size_t)8 * pa.nsplit * n * HT * hd * 2));
    VLA_TRY(al((void**)&pa.astat, (size_t)8 * pa.nsplit * n * HT * 2 * 4));
    VLA_TRY(al(&pa.omerged, (size_t)8 * n * HT * hd * 2));
    VLA_TRY(al(&pa.hbuf, (size_t)8 * n * (F / 8) * 2));
    VLA_TRY(al((void**)&pa.delta, (size_t)2 * 8 * n * d * 4));
    VLA_TRY(al((void**)&pa.sync, (size_t)PERSIST_SYNC_WORDS * 4));
    pa.err = reinterpret_cast<int*>(pa.sync + PERSIST_ERR_OFF);
    p->persist_err = pa.err;
    if (hipHostMalloc((void**)&p->persist_err_host, 16, hipHostMallocDefault) != hipSuccess) {
      p->persist_err_host = nullptr;
      return fail(VLA_E_NOMEM, "hipHostMalloc of the error word failed");
    }
    *p->persist_err_host = 0;
    VLA_TRY(al((void**)&p->trace, (size_t)8 * PERSIST_TRACE_MAX * 8));
    pa.trace = nullptr;
    const int* tracing = &m->trace;
    const long* spin = &m->spin_limit;
    int* err_host = p->persist_err_host;
    unsigned long long* tbuf = p->trace;
    // Per step and layer: the weights once, the cache once (algorithmic bytes).
    double wbytes = 0.0;
    for (int l = 0; l < L; ++l) {
      const SubW& at = m->layers[l][0];
      const SubW& ml = m->layers[l][1];
      wbytes += ((double)at.n_qkv * d + (double)d * dq + (double)(pa.glu ? 2 : 1) * F * d + (double)d * F) * es;
      (void)ml;
    }
    const double cbytes = (double)L * 2 * c.n_kv_heads * P * hd * es;
    const double gflop = (double)T * (2.0 * n * wbytes / es + 4.0 * n * c.n_heads * hd * (P + n) * L);
    // Every launch starts from cleared barrier flags, rank counters and error
    // word; the error word is copied to pinned host memory after the kernel,
    // where the next call (or vla_model_check) finds it.
    bld.ops->push_back(Op{[=](hipStream_t s) {
                            hipError_t e = launch_fill_u32(pa.sync, 0u, PERSIST_SYNC_WORDS, s);
                            if (e != hipSuccess) return e;
                            PersistArgs q = pa;
                            q.trace = *tracing ? tbuf : nullptr;
                            q.trace_all = *tracing == 2 ? 1 : 0;
                            q.spin_limit = *spin;
                            e = launch_persist(q, s);
                            if (e != hipSuccess) return e;
                            return hipMemcpyAsync(err_host, pa.err, 4, hipMemcpyDeviceToHost, s);
                          },
                          op_info(VLA_OP_PERSIST, n, L, T, (double)T * (wbytes + cbytes), gflop)});
    HIP_TRY(hipDeviceSynchronize());
    return VLA_OK;
  }

  // Residual projection (O or down) of a dense model: split-K partials summed
  // by the following row kernel (skinny), or the residual update in the
  // epilogue (wide).  Returns the partial count the row kernel must add.
  auto resid_gemm = [&](GemmArgs g, const float* alp, RowNormArgs& rn) {
    DenseLaunch dl;
    g.epi = EPI_PARTIAL;
    dl = dense_launch(et, g, 1);
    if (dl.skinny || (dl.tile && dl.tl.nsplit > 1)) {
      g.out = nullptr;  // set at run time from the plan's partial buffer
      g.ldo = d;
      part_need = std::max(part_need, (size_t)dl.splits() * M * d);
      GemmArgs gg = g;
      float** partp = &p->part;
      const double bytes = (double)g.N * g.K * es + (double)g.M * g.K * es + 4.0 * dl.splits() * g.M * g.N;
      bld.ops->push_back(Op{[=](hipStream_t s) {
                              GemmArgs q = gg;
                              q.out = *partp;
                              return launch_dense(et, dl, q, s);
                            },
                            op_info(VLA_OP_GEMM, g.M, g.N, g.K, bytes, 2.0 * g.M * g.N * g.K)});
      rn.nsplit = dl.splits();
      rn.alpha = alp;
    } else {
      g.epi = EPI_RESID;
      g.xres = p->x;
      g.ldxr = d;
      g.alpha = alp;
      bld.gemm(g, 1);
      rn.nsplit = 0;
      rn.alpha = nullptr;
    }
  };

  const size_t layer_block = (size_t)2 * B * c.n_kv_heads * P * hd;  // elements per cache layer
  for (int k = 0; k < T; ++k) {
    const float* modk = c.head_regression ? m->mod_static : p->mods + (size_t)k * modrow;
    const float* modfk = c.head_regression ? m->modf_static : p->modf + (size_t)k * 2 * d;
    // (gamma, beta) of the sublayer after (l, j); the final pair after the last one
    auto next_gb = [&](int l, int j, const float** gam, const float** bet) {
      int nl = l, nj = j + 1;
      if (nj >= (int)m->layers[l].size()) {
        nl = l + 1;
        nj = 0;
      }
      if (nl >= L) {
        *gam = modfk;
        *bet = modfk + d;
      } else {
        *gam = modk + ((size_t)nl * ns + nj) * 3 * d;
        *bet = *gam + d;
      }
    };
    RowNormArgs rn{};
    rn.mode = 1; rn.M = M; rn.d = d; rn.x = p->x; rn.a = p->a; rn.W_in = m->W_in; rn.xs = p->xs;
    rn.E_pos = m->E_pos; rn.n = nt; rn.stok = stok; rn.b_in = m->b_in; rn.A = A; rn.eps = c.rms_eps; rn.u = p->u; rn.u_f32 = u32;
    if (L > 0) {
      rn.gamma = modk;
      rn.beta = modk + d;
      if (m->tern) {  // the first sublayer's W2A8 input, quantised in the same kernel
        rn.q = p->q8;
        rn.qr = p->r8;
      }
    } else {
      rn.gamma = modfk;
      rn.beta = modfk + d;
      rn.u_f32 = et == ET_F32;
    }
    bld.row_norm(rn);
    for (int l = 0; l < L; ++l) {
      const std::vector<SubW>& subs = m->layers[l];
      for (int j = 0; j < (int)subs.size(); ++j) {
        const SubW& sw = subs[j];
        const float* alp = modk + ((size_t)l * ns + j) * 3 * d + 2 * d;
        RowNormArgs nr{};
        nr.mode = 0; nr.M = M; nr.d = d; nr.x = p->x; nr.eps = c.rms_eps; nr.u = p->u; nr.u_f32 = u32;
        next_gb(l, j, &nr.gamma, &nr.beta);
        // the head projection is dense: it reads u in the element type
        const bool last_sub = l == L - 1 && j == (int)subs.size() - 1;
        if (last_sub) nr.u_f32 = et == ET_F32;
        if (m->tern && !last_sub) {  // the next sublayer's W2A8 input
          nr.q = p->q8;
          nr.qr = p->r8;
        }
        if (sw.kind == K_MLP) {
          const bool glu = c.mlp != VLA_MLP_GELU;
          const int ngu = glu ? 2 * F : F;
          if (!m->tern) {
            GemmArgs g = gemm_base(m, M, ngu, d, p->u, d, sw.gu);
            g.epi = glu ? EPI_GLU : EPI_STORE;
            g.act = mlp_act(c.mlp);
            g.out = p->h;
            g.ldo = F;
            bld.gemm(g, glu ? 2 : 1);
            resid_gemm(gemm_base(m, M, d, F, p->h, F, sw.dn), alp, nr);
          } else {
            // u was quantised (q8, r8) by the row kernel that wrote it
            QuantArgs q{};
            TernArgs t{};
            t.M = M; t.N = ngu; t.K = d; t.x = p->q8; t.w = (const uint8_t*)sw.gu; t.rscale = p->r8; t.wscale = sw.s_gu;
            t.e = gemm_base(m, M, ngu, d, nullptr, 0, nullptr);
            t.e.epi = glu ? EPI_GLU : EPI_STORE;
            t.e.act = mlp_act(c.mlp);
            t.e.out = p->h;
            t.e.ldo = F;
            t.e.out_f32 = 1;
            bld.tern(t, glu ? 2 : 1);
            q = QuantArgs{};
            q.M = M; q.K = F; q.x = p->h; q.ldx = F; q.src_type = 0; q.q = p->q8; q.r = p->r8;
            bld.quant(q);
            t = TernArgs{};
            t.M = M; t.N = d; t.K = F; t.x = p->q8; t.w = (const uint8_t*)sw.dn; t.rscale = p->r8; t.wscale = sw.s_dn;
            t.e = gemm_base(m, M, d, F, nullptr, 0, nullptr);
            t.e.epi = EPI_RESID;
            t.e.xres = p->x;
            t.e.ldxr = d;
            t.e.alpha = alp;
            bld.tern(t, 1);
          }
        } else {
          if (!m->tern) {
            GemmArgs g = gemm_base(m, M, sw.n_qkv, d, p->u, d, sw.qkv);
            g.epi = EPI_STORE;
            g.out = p->qkv;
            g.ldo = ldqkv;
            bld.gemm(g, 1);
          } else {
            // u was quantised (q8, r8) by the row kernel that wrote it
            TernArgs t{};
            t.M = M; t.N = sw.n_qkv; t.K = d; t.x = p->q8; t.w = (const uint8_t*)sw.qkv; t.rscale = p->r8;
            t.wscale = sw.s_qkv;
            t.e = gemm_base(m, M, sw.n_qkv, d, nullptr, 0, nullptr);
            t.e.epi = EPI_STORE;
            t.e.out = p->qkv;
            t.e.ldo = ldqkv;
            bld.tern(t, 1);
          }
          if (m->rope_base > 0.0f && sw.kind != K_CROSS) {
            // RoPE variant: action token i at position i (self) or P + i (joint)
            void* qkvp = p->qkv;
            const int et = m->et, H = c.n_heads, G = c.n_kv_heads, pos0 = sw.kind == K_JOINT ? P : 0;
            const float base = m->rope_base;
            const double rb = 2.0 * M * (dq + dkv) * esize(et);
            bld.small([=](hipStream_t st) {
              hipError_t e = launch_rope(et, qkvp, M, nt, ldqkv, 0, H, hd, pos0, base, st);
              return e != hipSuccess ? e : launch_rope(et, qkvp, M, nt, ldqkv, dq, G, hd, pos0, base, st);
            }, M, dq + dkv, 0, rb);
          }
          AttnArgs at{};
          at.mode = sw.kind == K_SELF ? 0 : (sw.kind == K_CROSS ? 1 : 2);
          at.causal = (m->causal && sw.kind != K_CROSS) ? 1 : 0;
          at.B = B; at.n = nt; at.P = P; at.H = c.n_heads; at.G = c.n_kv_heads; at.hd = hd;
          at.q = p->qkv; at.ldq = ldqkv;
          at.ks = (const char*)p->qkv + (size_t)dq * es;
          at.vs = (const char*)p->qkv + (size_t)(dq + dkv) * es;
          at.ldkv = ldqkv;
          at.kc = nullptr;
          at.vc = nullptr;
          at.cp = cp;
          at.layer_off = sw.cache_idx >= 0 ? (size_t)sw.cache_idx * layer_block : 0;
          at.o = p->o;
          at.ldo = dq;
          at.scale = 1.0f / std::sqrt((float)hd);
          bld.attn(at);
          if (!m->tern) {
            resid_gemm(gemm_base(m, M, d, dq, p->o, dq, sw.o), alp, nr);
          } else {
            QuantArgs q{};
            q.M = M; q.K = dq; q.x = p->o; q.ldx = dq; q.src_type = 1; q.q = p->q8; q.r = p->r8;
            bld.quant(q);
            TernArgs t{};
            t.M = M; t.N = d; t.K = dq; t.x = p->q8; t.w = (const uint8_t*)sw.o; t.rscale = p->r8; t.wscale = sw.s_o;
            t.e = gemm_base(m, M, d, dq, nullptr, 0, nullptr);
            t.e.epi = EPI_RESID;
            t.e.xres = p->x;
            t.e.ldxr = d;
            t.e.alpha = alp;
            bld.tern(t, 1);
          }
        }
        // finish the residual stream and normalise for the next sublayer
        float** partp = &p->part;
        const double bytes = (double)M * d * (8.0 + 4.0 * std::min(nr.nsplit, 1) + (u32 ? 4.0 : es));
        bld.ops->push_back(Op{[=](hipStream_t s) {
                                RowNormArgs r = nr;
                                r.part = *partp;
                                return launch_row_norm(et, r, s);
                              },
                              op_info(VLA_OP_SMALL, M, d, nr.nsplit, bytes, 0.0)});
      }
    }
    // head: out-projection of the finally-normalised stream and the Euler update
    GemmArgs g = gemm_base(m, M, A, d, p->u, d, m->W_out);
    g.epi = EPI_EULER;
    g.bias = m->b_out;
    g.a = p->a;
    g.cp = cp;
    g.step = k;
    g.regression = c.head_regression;
    g.last = (k == T - 1);
    g.stok = stok;
    bld.gemm(g, 1);
  }

  if (part_need) VLA_TRY(al((void**)&p->part, part_need * 4));
  if (bld.part_need) VLA_TRY(al(&p->apart, bld.part_need));
  if (bld.stats_need) VLA_TRY(al((void**)&p->astats, bld.stats_need));
  HIP_TRY(hipDeviceSynchronize());
  return VLA_OK;
}

vla_status run_ops(const std::vector<Op>& ops, hipStream_t s) {
  for (const Op& op : ops) HIP_TRY(op(s));
  return VLA_OK;
}

// Launch-per-phase with a HIP event pair around every launch, each launch
// repeated `reps` times between its two events (the mean is elapsed / reps, so
// the cost of recording the events is amortised).  Repeated launches redo
// in-place updates, so a profiled call with reps > 1 is for timing only.
vla_status run_ops_profiled(Plan* p, hipStream_t s, int reps) {
  if (p->events.size() != 2 * p->ops.size()) {
    for (hipEvent_t e : p->events) (void)hipEventDestroy(e);
    p->events.assign(2 * p->ops.size(), nullptr);
    for (auto& e : p->events) HIP_TRY(hipEventCreate(&e));
  }
  for (size_t i = 0; i < p->ops.size(); ++i) {
    HIP_TRY(hipEventRecord(p->events[2 * i], s));
    for (int r = 0; r < reps; ++r) HIP_TRY(p->ops[i](s));
    HIP_TRY(hipEventRecord(p->events[2 * i + 1], s));
  }
  return VLA_OK;
}

}  // namespace

vla_model::~vla_model() {
  plans.clear();
  prefix_ws.clear();
  if (cap_stream) (void)hipStreamDestroy(cap_stream);
  for (void* p : allocs) (void)hipFree(p);
}

// ----------------------------------------------------------------------------
// C ABI

extern "C" {

const char* vla_last_error(void) { return g_err.c_str(); }

const char* vla_status_string(int32_t st) {
  switch (st) {
    case VLA_OK: return "VLA_OK";
    case VLA_E_ARG: return "VLA_E_ARG";
    case VLA_E_SHAPE: return "VLA_E_SHAPE";
    case VLA_E_UNSUPPORTED: return "VLA_E_UNSUPPORTED";
    case VLA_E_NOMEM: return "VLA_E_NOMEM";
    case VLA_E_DEVICE: return "VLA_E_DEVICE";
    case VLA_E_NONFINITE: return "VLA_E_NONFINITE";
  }
  return "unknown status";
}

int32_t vla_weight_count(const vla_config* c) {
  if (validate_config(c) != VLA_OK) return -1;
  const bool tern = c->wtype == VLA_W_TERNARY;
  const int per_mat = tern ? 2 : 1;
  int cnt = 5 + (c->head_regression ? 1 : 6) + 2;
  for (int l = 0; l < c->n_layers; ++l) {
    cnt += c->head_regression ? 1 : 2;
    for (int k : sublayers(*c, l)) {
      if (k == K_MLP) {
        cnt += (c->mlp == VLA_MLP_GELU ? 2 : 3) * per_mat;
      } else {
        cnt += 2 * per_mat;                          // W_q, W_o
        if (has_self(k)) cnt += 2 * per_mat;         // W_k, W_v
        if (has_prefix(k)) cnt += 2 * per_mat;       // W_kc, W_vc
      }
    }
  }
  return cnt;
}

vla_status vla_model_set_option(vla_model* m, int32_t option, int32_t value) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  if (option == VLA_OPT_LOOP_MODE) {
    if (value < 0 || value > 2) return fail(VLA_E_ARG, "loop mode %d out of range", value);
    m->loop_mode = value;
    return VLA_OK;
  }
  if (option == VLA_OPT_ATTN_SPLITS) {
    if (value < 0 || value % 100 > 64 || value / 100 > 8)
      return fail(VLA_E_ARG, "attention splits %d out of range", value);
    if (value != m->attn_splits) {
      m->plans.clear();            // plans bake the split count in
      m->last_profiled = nullptr;
      m->last_traced = nullptr;
    }
    m->attn_splits = value;
    return VLA_OK;
  }
  if (option == VLA_OPT_ROPE_BASE) {
    if (value < 0 || value == 1 || value > 10000000) return fail(VLA_E_ARG, "RoPE base %d out of range", value);
    if ((float)value != m->rope_base) {
      m->plans.clear();            // plans bake the rotation in
      m->last_profiled = nullptr;
      m->last_traced = nullptr;
    }
    m->rope_base = (float)value;
    return VLA_OK;
  }
  if (option == VLA_OPT_STATE_TOKEN) {
    if (value < 0 || value > 1) return fail(VLA_E_ARG, "state-token flag %d out of range", value);
    if (value != m->state_token) {
      m->plans.clear();            // plans bake the row count and the loop driver in
      m->last_profiled = nullptr;
      m->last_traced = nullptr;
    }
    m->state_token = value;
    return VLA_OK;
  }
  if (option == VLA_OPT_CAUSAL_SELF) {
    if (value < 0 || value > 1) return fail(VLA_E_ARG, "causal flag %d out of range", value);
    if (value != m->causal) {
      m->plans.clear();            // plans bake the mask and the loop driver in
      m->last_profiled = nullptr;
      m->last_traced = nullptr;
    }
    m->causal = value;
    return VLA_OK;
  }
  if (option == VLA_OPT_PERSIST_SPIN_LIMIT) {
    if (value < -1) return fail(VLA_E_ARG, "spin limit %d out of range", value);
    m->spin_limit = value < 0 ? PERSIST_SPIN_DEFAULT : (long)value;
    return VLA_OK;
  }
  if (option == VLA_OPT_TRACE) {
    if (value < 0 || value > 2) return fail(VLA_E_ARG, "trace mode %d out of range", value);
    m->trace = value;
    return VLA_OK;
  }
  if (option == VLA_OPT_PROFILE) {
    if (value < 0 || value > 1000) return fail(VLA_E_ARG, "profile repetitions %d out of range", value);
    m->profile = value;
    return VLA_OK;
  }
  return fail(VLA_E_ARG, "unknown option %d", option);
}

void vla_model_destroy(vla_model* m) { delete m; }

vla_status vla_model_check(vla_model* m, void* stream) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  const hipError_t e = hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(VLA_E_DEVICE, "hipStreamSynchronize: %s", hipGetErrorString(e));
  return take_device_error(m);
}

size_t vla_kv_cache_bytes(const vla_model* m, int32_t batch, int32_t prefix_len) {
  if (!m || batch < 1 || prefix_len < 1) return 0;
  return (size_t)m->Lc * 2 * batch * m->cfg.n_kv_heads * (size_t)prefix_len * m->cfg.head_dim * esize(m->et);
}

}  // extern "C"

namespace {

// Device copy of one table matrix into library memory.
vla_status copy_in(vla_model* m, void** dst, const void* src, size_t bytes) {
  Alloc al{m->allocs};
  VLA_TRY(al(dst, bytes));
  HIP_TRY(hipMemcpy(*dst, src, bytes, hipMemcpyDeviceToDevice));
  return VLA_OK;
}

// Copies rows of `src` ([rows][rowbytes]) into dst rows dst_row0 + 32*blk + (0..15)
// for each 16-row block blk (gate/up interleave); plain copy when interleave is false.
vla_status copy_rows(void* dst, size_t dst_row0, const void* src, int rows, size_t rowbytes, bool interleave) {
  char* d = (char*)dst + dst_row0 * rowbytes;
  if (!interleave) {
    HIP_TRY(hipMemcpy(d, src, (size_t)rows * rowbytes, hipMemcpyDeviceToDevice));
    return VLA_OK;
  }
  HIP_TRY(hipMemcpy2D(d, 32 * rowbytes, src, 16 * rowbytes, 16 * rowbytes, rows / 16, hipMemcpyDeviceToDevice));
  return VLA_OK;
}

float read_scale(const void* p, vla_status* st) {
  float v = 0.0f;
  if (hipMemcpy(&v, p, 4, hipMemcpyDeviceToHost) != hipSuccess) *st = fail(VLA_E_DEVICE, "reading a ternary scale failed");
  else if (!std::isfinite(v)) *st = fail(VLA_E_ARG, "ternary scale is not finite");
  return v;
}

vla_status upload_scales(vla_model* m, float** dst, const std::vector<float>& v) {
  Alloc al{m->allocs};
  VLA_TRY(al((void**)dst, v.size() * 4));
  HIP_TRY(hipMemcpy(*dst, v.data(), v.size() * 4, hipMemcpyHostToDevice));
  return VLA_OK;
}

// A group of matrices fused along rows: dense or packed.
struct Part {
  const void* src;
  int rows;
  float scale;
};

vla_status fuse(vla_model* m, void** dst, float** scales, const std::vector<Part>& parts, int K, bool interleave) {
  const bool tern = m->tern;
  const size_t rowbytes = tern ? (size_t)K / 4 : (size_t)K * esize(m->et);
  int rows = 0;
  for (auto& p : parts) rows += p.rows;
  Alloc al{m->allocs};
  VLA_TRY(al(dst, (size_t)rows * rowbytes));
  std::vector<float> sc;
  if (interleave) {
    // two parts of equal rows: blocks of 16 rows alternate between them
    VLA_TRY(copy_rows(*dst, 0, parts[0].src, parts[0].rows, rowbytes, true));
    VLA_TRY(copy_rows(*dst, 16, parts[1].src, parts[1].rows, rowbytes, true));
    for (int b = 0; b < parts[0].rows / 16; ++b) {
      for (int i = 0; i < 16; ++i) sc.push_back(parts[0].scale);
      for (int i = 0; i < 16; ++i) sc.push_back(parts[1].scale);
    }
  } else {
    size_t r0 = 0;
    for (auto& p : parts) {
      VLA_TRY(copy_rows(*dst, r0, p.src, p.rows, rowbytes, false));
      r0 += p.rows;
      for (int i = 0; i < p.rows; ++i) sc.push_back(p.scale);
    }
  }
  if (tern && scales) VLA_TRY(upload_scales(m, scales, sc));
  return VLA_OK;
}

vla_status create_impl(const vla_config* cfg, const void* const* weights, int32_t n_weights, vla_model** out) {
  const vla_config& c = *cfg;
  std::unique_ptr<vla_model> m(new vla_model());
  m->cfg = c;
  m->tern = c.wtype == VLA_W_TERNARY;
  m->et = c.wtype == VLA_W_F32 ? ET_F32 : ET_BF16;
  m->d = c.d_model;
  m->dq = c.n_heads * c.head_dim;
  m->dkv = c.n_kv_heads * c.head_dim;
  m->ns = n_sub(c);
  m->Lc = cache_layers(c);
  const int d = m->d, A = c.d_action, S = c.d_state, n = c.n_action, F = c.d_ff, dp = c.d_prefix;
  const int dq = m->dq, dkv = m->dkv, ns = m->ns, L = c.n_layers;
  const size_t es = esize(m->et);
  TableReader tr{weights, n_weights};
  const void* p;
  Alloc al{m->allocs};

  VLA_TRY(tr.next(&p, "W_in")); VLA_TRY(copy_in(m.get(), &m->W_in, p, (size_t)d * A * es));
  VLA_TRY(tr.next(&p, "b_in")); VLA_TRY(copy_in(m.get(), (void**)&m->b_in, p, (size_t)d * 4));
  if (S > 0) {
    VLA_TRY(tr.next(&p, "W_s")); VLA_TRY(copy_in(m.get(), &m->W_s, p, (size_t)d * S * es));
  } else {
    VLA_TRY(tr.next(&p, "W_s")); VLA_TRY(al(&m->W_s, 16));
  }
  VLA_TRY(tr.next(&p, "b_s")); VLA_TRY(copy_in(m.get(), (void**)&m->b_s, p, (size_t)d * 4));
  VLA_TRY(tr.next(&p, "E_pos")); VLA_TRY(copy_in(m.get(), &m->E_pos, p, (size_t)n * d * es));
  if (c.head_regression) {
    VLA_TRY(tr.next(&p, "mod_f")); VLA_TRY(copy_in(m.get(), (void**)&m->modf_static, p, (size_t)2 * d * 4));
  } else {
    VLA_TRY(tr.next(&p, "W_t1")); VLA_TRY(copy_in(m.get(), &m->W_t1, p, (size_t)d * d * es));
    VLA_TRY(tr.next(&p, "b_t1")); VLA_TRY(copy_in(m.get(), (void**)&m->b_t1, p, (size_t)d * 4));
    VLA_TRY(tr.next(&p, "W_t2")); VLA_TRY(copy_in(m.get(), &m->W_t2, p, (size_t)d * d * es));
    VLA_TRY(tr.next(&p, "b_t2")); VLA_TRY(copy_in(m.get(), (void**)&m->b_t2, p, (size_t)d * 4));
    VLA_TRY(tr.next(&p, "W_fm")); VLA_TRY(copy_in(m.get(), &m->W_fm, p, (size_t)2 * d * d * es));
    VLA_TRY(tr.next(&p, "b_fm")); VLA_TRY(copy_in(m.get(), (void**)&m->b_fm, p, (size_t)2 * d * 4));
  }
  VLA_TRY(tr.next(&p, "W_out")); VLA_TRY(copy_in(m.get(), &m->W_out, p, (size_t)A * d * es));
  VLA_TRY(tr.next(&p, "b_out")); VLA_TRY(copy_in(m.get(), (void**)&m->b_out, p, (size_t)A * 4));

  const size_t modrow = (size_t)3 * ns * d;
  if (c.head_regression) {
    VLA_TRY(al((void**)&m->mod_static, (size_t)L * modrow * 4));
  } else {
    VLA_TRY(al(&m->W_mod, (size_t)L * modrow * d * es));
    VLA_TRY(al((void**)&m->b_mod, (size_t)L * modrow * 4));
  }

  auto mat = [&](const char* what, const void** src, float* scale) -> vla_status {
    VLA_TRY(tr.next(src, what));
    if (m->tern) {
      const void* sp;
      VLA_TRY(tr.next(&sp, "ternary scale"));
      vla_status st = VLA_OK;
      *scale = read_scale(sp, &st);
      return st;
    }
    *scale = 1.0f;
    return VLA_OK;
  };

  int cidx = 0;
  m->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    if (c.head_regression) {
      VLA_TRY(tr.next(&p, "mod"));
      HIP_TRY(hipMemcpy((char*)m->mod_static + (size_t)l * modrow * 4, p, modrow * 4, hipMemcpyDeviceToDevice));
    } else {
      VLA_TRY(tr.next(&p, "W_mod"));
      HIP_TRY(hipMemcpy((char*)m->W_mod + (size_t)l * modrow * d * es, p, modrow * d * es, hipMemcpyDeviceToDevice));
      VLA_TRY(tr.next(&p, "b_mod"));
      HIP_TRY(hipMemcpy((char*)m->b_mod + (size_t)l * modrow * 4, p, modrow * 4, hipMemcpyDeviceToDevice));
    }
    for (int k : sublayers(c, l)) {
      SubW sw;
      sw.kind = k;
      if (k == K_MLP) {
        if (c.mlp == VLA_MLP_GELU) {
          const void *w1, *w2;
          float s1, s2;
          VLA_TRY(mat("W1", &w1, &s1));
          VLA_TRY(mat("W2", &w2, &s2));
          VLA_TRY(fuse(m.get(), &sw.gu, &sw.s_gu, {{w1, F, s1}}, d, false));
          VLA_TRY(fuse(m.get(), &sw.dn, &sw.s_dn, {{w2, d, s2}}, F, false));
        } else {
          const void *wg, *wu, *wd;
          float sg, su, sd;
          VLA_TRY(mat("W_g", &wg, &sg));
          VLA_TRY(mat("W_u", &wu, &su));
          VLA_TRY(mat("W_d", &wd, &sd));
          VLA_TRY(fuse(m.get(), &sw.gu, &sw.s_gu, {{wg, F, sg}, {wu, F, su}}, d, true));
          VLA_TRY(fuse(m.get(), &sw.dn, &sw.s_dn, {{wd, d, sd}}, F, false));
        }
      } else {
        const void *wq, *wk = nullptr, *wv = nullptr, *wkc = nullptr, *wvc = nullptr, *wo;
        float sq, sk = 1, sv = 1, skc = 1, svc = 1, so;
        VLA_TRY(mat("W_q", &wq, &sq));
        if (has_self(k)) {
          VLA_TRY(mat("W_k", &wk, &sk));
          VLA_TRY(mat("W_v", &wv, &sv));
        }
        if (has_prefix(k)) {
          VLA_TRY(mat("W_kc", &wkc, &skc));
          VLA_TRY(mat("W_vc", &wvc, &svc));
        }
        VLA_TRY(mat("W_o", &wo, &so));
        std::vector<Part> qkv = {{wq, dq, sq}};
        if (has_self(k)) {
          qkv.push_back({wk, dkv, sk});
          qkv.push_back({wv, dkv, sv});
        }
        sw.n_qkv = has_self(k) ? dq + 2 * dkv : dq;
        VLA_TRY(fuse(m.get(), &sw.qkv, &sw.s_qkv, qkv, d, false));
        if (has_prefix(k)) {
          VLA_TRY(fuse(m.get(), &sw.kvc, &sw.s_kvc, {{wkc, dkv, skc}, {wvc, dkv, svc}}, dp, false));
          sw.cache_idx = cidx++;
        }
        VLA_TRY(fuse(m.get(), &sw.o, &sw.s_o, {{wo, d, so}}, dq, false));
      }
      m->layers[l].push_back(sw);
    }
  }
  if (tr.i != n_weights)
    return fail(VLA_E_ARG, "weight table has %d entries, expected %d", n_weights, tr.i);
  if (!m->tern && cidx > 0) {
    // one [Lc * 2 d_kv][d_p] matrix so that the prefix build is a single GEMM
    const size_t slot_bytes = (size_t)2 * dkv * dp * es;
    VLA_TRY(al(&m->kvc_all, (size_t)cidx * slot_bytes));
    for (auto& lay : m->layers)
      for (auto& sw : lay)
        if (sw.cache_idx >= 0)
          HIP_TRY(hipMemcpy((char*)m->kvc_all + (size_t)sw.cache_idx * slot_bytes, sw.kvc, slot_bytes,
                            hipMemcpyDeviceToDevice));
  }
  HIP_TRY(hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking));
  HIP_TRY(hipDeviceSynchronize());
  *out = m.release();
  return VLA_OK;
}

vla_status get_prefix_ws(vla_model* m, int B, int P, PrefixWs** out) {
  auto key = std::make_pair(B, P);
  auto it = m->prefix_ws.find(key);
  if (it != m->prefix_ws.end()) {
    *out = it->second.get();
    return VLA_OK;
  }
  std::unique_ptr<PrefixWs> w(new PrefixWs());
  if (m->tern) {
    Alloc al{w->allocs};
    const size_t M = (size_t)B * P;
    VLA_TRY(al((void**)&w->q8, M * m->cfg.d_prefix));
    VLA_TRY(al((void**)&w->r8, M * 4));
    HIP_TRY(hipDeviceSynchronize());
  }
  *out = w.get();
  m->prefix_ws[key] = std::move(w);
  return VLA_OK;
}

bool env_flag(const char* name) {
  const char* v = std::getenv(name);
  return v && v[0] == '1';
}

}  // namespace

extern "C" {

vla_status vla_model_create(const vla_config* cfg, const void* const* weights, int32_t n_weights, vla_model** out) {
  if (!out) return fail(VLA_E_ARG, "out is NULL");
  *out = nullptr;
  VLA_TRY(validate_config(cfg));
  if (!weights) return fail(VLA_E_ARG, "weight table is NULL");
  const int32_t want = vla_weight_count(cfg);
  if (n_weights != want) return fail(VLA_E_ARG, "weight table has %d entries, expected %d", n_weights, want);
  return create_impl(cfg, weights, n_weights, out);
}

}  // extern "C"

// RoPE variant: the cached K of every joint layer holds prefix row p at
// position p (cache block [2][B][G][P][hd], K first).
// Device scratch of the no-allocation prefix build: one copy per GPU, held
// until the process ends.  Host code must not use the symbol itself as an
// address: prefix_scratch() returns the device's copy, looked up once per
// device with hipGetSymbolAddress.
constexpr size_t kPrefixScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char prefix_scratch_buf[kPrefixScratchBytes];

static vla_status prefix_scratch(unsigned char** out) {
  static std::mutex mu;
  static unsigned char* ptr[64] = {};
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(VLA_E_UNSUPPORTED, "device %d beyond 64", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(prefix_scratch_buf));
    if (e != hipSuccess || !p)
      return fail(VLA_E_DEVICE, "hipGetSymbolAddress of the prefix scratch: %s", hipGetErrorString(e));
    ptr[dev] = static_cast<unsigned char*>(p);
  }
  *out = ptr[dev];
  return VLA_OK;
}

static vla_status check_prefix_args(vla_model* m, const void* prefix_hidden, int batch, int prefix_len,
                                    const void* kv_cache, size_t kv_cache_bytes) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  if (!prefix_hidden || !kv_cache) return fail(VLA_E_ARG, "prefix_hidden / kv_cache is NULL");
  if (!al16(prefix_hidden) || !al16(kv_cache)) return fail(VLA_E_ARG, "buffers must be 16-byte aligned");
  if (batch < 1 || prefix_len < 1) return fail(VLA_E_SHAPE, "batch and prefix_len must be >= 1");
  if ((long long)batch * prefix_len > (1LL << 24)) return fail(VLA_E_UNSUPPORTED, "batch * prefix_len too large");
  if (kv_cache_bytes != vla_kv_cache_bytes(m, batch, prefix_len))
    return fail(VLA_E_SHAPE, "kv_cache_bytes %zu != %zu for batch %d, prefix_len %d", kv_cache_bytes,
                vla_kv_cache_bytes(m, batch, prefix_len), batch, prefix_len);
  return VLA_OK;
}

static vla_status rope_prefix(vla_model* m, void* kv_cache, int batch, int prefix_len, size_t layer_block,
                              hipStream_t s) {
  if (m->rope_base <= 0.0f) return VLA_OK;
  const size_t es = m->et == ET_BF16 ? 2 : 4;
  for (auto& lay : m->layers)
    for (auto& sw : lay) {
      if (sw.cache_idx < 0 || sw.kind != K_JOINT) continue;
      void* kb = (char*)kv_cache + (size_t)sw.cache_idx * layer_block * es;
      const int rows = batch * m->cfg.n_kv_heads * prefix_len;
      HIP_TRY(launch_rope(m->et, kb, rows, prefix_len, m->cfg.head_dim, 0, 1, m->cfg.head_dim, 0, m->rope_base, s));
    }
  return VLA_OK;
}

// The prefix build proper: quantise the prefix rows into (q8, r8) for W2A8
// models, then one GEMM over every layer's stacked cross K/V weights (dense)
// or one W2A8 GEMM per layer, with the cache-slot epilogue; RoPE variant last.
static vla_status prefix_kv_build_impl(vla_model* m, const void* prefix_hidden, int batch, int prefix_len,
                                       void* kv_cache, int8_t* q8, float* r8, hipStream_t s) {
  const int M = batch * prefix_len, N = 2 * m->dkv, K = m->cfg.d_prefix, hd = m->cfg.head_dim;
  const size_t layer_block = (size_t)2 * batch * m->cfg.n_kv_heads * prefix_len * hd;
  const size_t es = esize(m->et);
  if (m->tern) {
    QuantArgs q{};
    q.M = M; q.K = K; q.x = prefix_hidden; q.ldx = K; q.src_type = 1; q.q = q8; q.r = r8;
    HIP_TRY(launch_quantize(q, s));
  }
  if (m->kvc_all) {
    // every layer's cross K/V in one GEMM: column n of slot n / (2 d_kv)
    GemmArgs g{};
    g.M = M; g.N = N * m->Lc; g.K = K; g.X = prefix_hidden; g.ldx = K; g.W = m->kvc_all;
    g.epi = EPI_KVCACHE;
    g.cache = kv_cache;
    g.P = prefix_len; g.hd = hd; g.d_kv = m->dkv; g.B = batch;
    g.lay_cols = N;
    g.lay_stride = layer_block;
    HIP_TRY(launch_dense(m->et, dense_launch(m->et, g, 1), g, s));
    return rope_prefix(m, kv_cache, batch, prefix_len, layer_block, s);
  }
  for (auto& lay : m->layers)
    for (auto& sw : lay) {
      if (sw.cache_idx < 0) continue;
      GemmArgs g{};
      g.M = M; g.N = N; g.K = K; g.X = prefix_hidden; g.ldx = K; g.W = sw.kvc;
      g.epi = EPI_KVCACHE;
      g.cache = (char*)kv_cache + (size_t)sw.cache_idx * layer_block * es;
      g.P = prefix_len; g.hd = hd; g.d_kv = m->dkv; g.B = batch;
      if (!m->tern) {
        HIP_TRY(launch_dense(m->et, dense_launch(m->et, g, 1), g, s));
      } else {
        TernArgs ta{};
        const Tiling t = tern_tiling(M, N, K, 1);
        ta.M = M; ta.N = N; ta.K = K; ta.x = q8; ta.w = (const uint8_t*)sw.kvc; ta.rscale = r8;
        ta.wscale = sw.s_kvc; ta.ks = t.nc * 256; ta.nsplit = 1; ta.n_tiles = t.n_tiles; ta.e = g;
        HIP_TRY(launch_ternary_gemm(ta, t.ms, t.units, s));
      }
    }
  return rope_prefix(m, kv_cache, batch, prefix_len, layer_block, s);
}

extern "C" {

vla_status vla_prefix_kv_build(vla_model* m, const void* prefix_hidden, int32_t batch, int32_t prefix_len,
                               void* kv_cache, size_t kv_cache_bytes, void* stream) {
  VLA_TRY(check_prefix_args(m, prefix_hidden, batch, prefix_len, kv_cache, kv_cache_bytes));
  PrefixWs* w = nullptr;
  VLA_TRY(get_prefix_ws(m, batch, prefix_len, &w));
  return prefix_kv_build_impl(m, prefix_hidden, batch, prefix_len, kv_cache, w->q8, w->r8,
                              reinterpret_cast<hipStream_t>(stream));
}

vla_status vla_prefix_kv_build_noalloc(vla_model* m, const void* prefix_hidden, int32_t batch, int32_t prefix_len,
                                       void* kv_cache, size_t kv_cache_bytes, void* stream) {
  VLA_TRY(check_prefix_args(m, prefix_hidden, batch, prefix_len, kv_cache, kv_cache_bytes));
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  if (m->tern) {
    // codes [M][d_p] int8, then the per-row absmax [M] fp32 at the next 256-byte boundary
    const size_t M = (size_t)batch * prefix_len;
    const size_t qbytes = (M * m->cfg.d_prefix + 255) / 256 * 256;
    if (qbytes + M * 4 > kPrefixScratchBytes)
      return fail(VLA_E_UNSUPPORTED, "batch * prefix_len * (d_prefix + 4) needs %zu bytes of scratch, more than "
                                     "the %zu of the no-allocation entry", qbytes + M * 4, kPrefixScratchBytes);
    unsigned char* base = nullptr;
    VLA_TRY(prefix_scratch(&base));
    q8 = reinterpret_cast<int8_t*>(base);
    r8 = reinterpret_cast<float*>(base + qbytes);
  }
  return prefix_kv_build_impl(m, prefix_hidden, batch, prefix_len, kv_cache, q8, r8,
                              reinterpret_cast<hipStream_t>(stream));
}

vla_status vla_denoise(vla_model* m, const void* kv_cache, size_t kv_cache_bytes, int32_t batch, int32_t prefix_len,
                       const float* noise, const float* state, const float* t_schedule, int32_t n_steps,
                       const float* act_mean, const float* act_std, float* actions_out, void* stream) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  const vla_config& c = m->cfg;
  if (!kv_cache || !noise || !actions_out || !t_schedule) return fail(VLA_E_ARG, "NULL buffer");
  if (c.d_state > 0 && !state) return fail(VLA_E_ARG, "state is NULL");
  for (const void* q : {kv_cache, (const void*)noise, (const void*)state, (const void*)act_mean, (const void*)act_std,
                        (const void*)actions_out})
    if (q && !al16(q)) return fail(VLA_E_ARG, "device buffers must be 16-byte aligned");
  if (batch < 1 || prefix_len < 1) return fail(VLA_E_SHAPE, "batch and prefix_len must be >= 1");
  const int ntok = c.n_action + (m->state_token ? 1 : 0);   // token rows per request
  if ((long long)batch * ntok > 65536) return fail(VLA_E_UNSUPPORTED, "batch * tokens too large");
  if ((prefix_len + 31) / 32 + (ntok + 31) / 32 > attention_max_blocks())
    return fail(VLA_E_UNSUPPORTED, "prefix_len + tokens beyond %d keys", 32 * attention_max_blocks() - 32);
  if (n_steps < 1 || n_steps > VLA_MAX_STEPS) return fail(VLA_E_SHAPE, "n_steps %d not in 1..%d", n_steps, VLA_MAX_STEPS);
  if (c.head_regression && n_steps != 1) return fail(VLA_E_SHAPE, "the regression head takes n_steps == 1");
  if (kv_cache_bytes != vla_kv_cache_bytes(m, batch, prefix_len))
    return fail(VLA_E_SHAPE, "kv_cache_bytes %zu != %zu for batch %d, prefix_len %d", kv_cache_bytes,
                vla_kv_cache_bytes(m, batch, prefix_len), batch, prefix_len);
  VLA_TRY(take_device_error(m));
  CallParams cpv{};
  for (int k = 0; k <= n_steps; ++k) {
    if (!std::isfinite(t_schedule[k])) return fail(VLA_E_ARG, "t_schedule[%d] is not finite", k);
    cpv.tau[k] = t_schedule[k];
  }
  cpv.kv_cache = kv_cache;
  cpv.noise = noise;
  cpv.state = state;
  cpv.actions_out = actions_out;
  cpv.act_mean = act_mean;
  cpv.act_std = act_std;

  const bool persist = m->loop_mode == 2 && persist_eligible(m, batch, prefix_len, n_steps);
  auto key = std::make_tuple(batch, prefix_len, n_steps, (int)persist);
  auto it = m->plans.find(key);
  Plan* p;
  if (it == m->plans.end()) {
    if (m->plans.size() >= 8) {
      if (m->last_profiled == m->plans.begin()->second.get()) m->last_profiled = nullptr;
      if (m->last_traced == m->plans.begin()->second.get()) m->last_traced = nullptr;
      m->plans.erase(m->plans.begin());
    }
    std::unique_ptr<Plan> np(new Plan());
    np->B = batch;
    np->P = prefix_len;
    np->T = n_steps;
    np->persist = persist;
    VLA_TRY(build_plan(m, np.get()));
    p = np.get();
    m->plans[key] = std::move(np);
  } else {
    p = it->second.get();
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(launch_set_params(p->cp, cpv, s));
  if (p->persist && m->trace) m->last_traced = p;
  if (m->profile) {
    VLA_TRY(run_ops_profiled(p, s, m->profile));
    m->last_profiled = p;
    p->prof_reps = m->profile;
  } else if (m->loop_mode == 0 || p->persist) {
    VLA_TRY(run_ops(p->ops, s));
  } else {
    if (!p->exec) {
      hipGraph_t graph = nullptr;
      HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeRelaxed));
      vla_status st = run_ops(p->ops, m->cap_stream);
      hipError_t e = hipStreamEndCapture(m->cap_stream, &graph);
      if (st != VLA_OK) {
        if (graph) (void)hipGraphDestroy(graph);
        return st;
      }
      if (e != hipSuccess) return fail(VLA_E_DEVICE, "hipStreamEndCapture: %s", hipGetErrorString(e));
      e = hipGraphInstantiate(&p->exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (e != hipSuccess) {
        p->exec = nullptr;
        return fail(VLA_E_DEVICE, "hipGraphInstantiate: %s", hipGetErrorString(e));
      }
    }
    HIP_TRY(hipGraphLaunch(p->exec, s));
  }
  if (env_flag("VLA_CHECK_FINITE")) {
    int* flag = nullptr;
    HIP_TRY(hipMalloc(&flag, 4));
    (void)hipMemsetAsync(flag, 0, 4, s);
    (void)launch_check_finite(actions_out, (size_t)batch * c.n_action * c.d_action, flag, s);
    int h = 0;
    (void)hipMemcpyAsync(&h, flag, 4, hipMemcpyDeviceToHost, s);
    hipError_t e = hipStreamSynchronize(s);
    (void)hipFree(flag);
    if (e != hipSuccess) return fail(VLA_E_DEVICE, "hipStreamSynchronize: %s", hipGetErrorString(e));
    VLA_TRY(take_device_error(m));   // a timed-out barrier also leaves NaN: name the cause first
    if (h) return fail(VLA_E_NONFINITE, "non-finite value in the action chunk");
  }
  return VLA_OK;
}

vla_status vla_ternary_gemm(const int8_t* x, const uint8_t* w_packed, int32_t M, int32_t N, int32_t K,
                            int32_t* acc_out, void* stream) {
  if (M < 0 || N < 0 || K < 0) return fail(VLA_E_SHAPE, "negative dimension");
  if (K % 4) return fail(VLA_E_SHAPE, "K %% 4 != 0");
  if (K > (1 << 23) / 128) return fail(VLA_E_SHAPE, "K too large for an exact int32 accumulator");
  if ((long long)M * N == 0) return VLA_OK;
  if (K > 0 && (!x || !w_packed)) return fail(VLA_E_ARG, "NULL input");
  if (!acc_out) return fail(VLA_E_ARG, "acc_out is NULL");
  if ((x && !al16(x)) || (w_packed && !al16(w_packed)) || !al16(acc_out))
    return fail(VLA_E_ARG, "buffers must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (K == 0) {
    HIP_TRY(launch_fill_u32(reinterpret_cast<unsigned*>(acc_out), 0u, (size_t)M * N, s));
    return VLA_OK;
  }
  TernArgs a{};
  a.M = M; a.N = N; a.K = K; a.x = x; a.w = w_packed; a.acc_out = acc_out;
  Tiling t = tern_tiling(M, N, K, 1);
  if (K % 64 != 0) t = Tiling{1, 1, 1, 1, 1, 1, 1};
  // Few output tiles: split K across workgroups; the int32 partial sums are
  // exact and are added atomically into the zero-filled output.
  if (!tern_tile_eligible(M, N, K) && K % 64 == 0 && t.units < 256 && K > 256) {
    t.nc = 1;
    t.nsplit = std::min(cdiv(K, 256), cdiv(256, t.units));
    while ((long long)t.nc * 256 * t.nsplit < K) ++t.nsplit;
    t.units *= t.nsplit;
  }
  a.ks = t.nc * 256; a.nsplit = t.nsplit; a.n_tiles = t.n_tiles;
  if (a.nsplit > 1) HIP_TRY(launch_fill_u32(reinterpret_cast<unsigned*>(acc_out), 0u, (size_t)M * N, s));
  HIP_TRY(launch_ternary_gemm(a, t.ms, t.units, s));
  return VLA_OK;
}

int32_t vla_profile_read(vla_model* m, vla_op_time* out, int32_t max_ops) {
  if (!m || !m->last_profiled) return -1;
  Plan* p = static_cast<Plan*>(m->last_profiled);
  const int32_t n = (int32_t)p->ops.size();
  for (int32_t i = 0; i < n && i < max_ops && out; ++i) {
    out[i] = p->ops[i].info;
    float ms = -1.0f;
    if (hipEventSynchronize(p->events[2 * i + 1]) == hipSuccess &&
        hipEventElapsedTime(&ms, p->events[2 * i], p->events[2 * i + 1]) != hipSuccess)
      ms = -1.0f;
    out[i].ms = ms < 0.0f ? ms : ms / (float)p->prof_reps;
  }
  return n;
}

// ---- test entries ----------------------------------------------------------

int32_t vla_test_persist_trace(vla_model* m, uint64_t* out, int32_t max_per_team) {
  if (!m || !m->last_traced) return -1;
  Plan* p = static_cast<Plan*>(m->last_traced);
  if (!p->trace || max_per_team < 0) return -1;
  if (hipDeviceSynchronize() != hipSuccess) return -1;
  const bool all = m->trace == 2;
  const int rows = all ? 256 : 8, cap = all ? PERSIST_TRACE_WG : PERSIST_TRACE_MAX;
  const int n = std::min(max_per_team, cap);
  if (out)
    for (int t = 0; t < rows; ++t)
      if (hipMemcpy(out + (size_t)t * n, p->trace + (size_t)t * cap, (size_t)n * 8, hipMemcpyDeviceToHost) != hipSuccess)
        return -1;
  return n;
}

vla_status vla_test_gemm(int32_t elem, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                         int32_t variant, float* y, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  if (variant < 0 || (variant > 4 && variant < 10) || variant > 14)
    return fail(VLA_E_ARG, "variant must be 0..4 or 10..14");
  if (!x || !w || !y || !al16(x) || !al16(w) || !al16(y)) return fail(VLA_E_ARG, "bad buffer");
  if (M < 1 || N < 1 || K < 1 || K % (elem ? 8 : 4)) return fail(VLA_E_SHAPE, "bad GEMM shape");
  const int et = elem ? ET_BF16 : ET_F32;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  GemmArgs g{};
  g.M = M; g.N = N; g.K = K; g.X = x; g.ldx = K; g.W = w;
  g.epi = EPI_STORE; g.out = y; g.ldo = N; g.out_f32 = 1;
  if (variant == 4) {
    // the residual projections' launch: split-K fp32 partials, summed here
    g.epi = EPI_PARTIAL;
    const DenseLaunch d = dense_launch(et, g, 1, 0);
    if (!d.skinny && !d.tile) return fail(VLA_E_UNSUPPORTED, "no split-K launch for this shape");
    float* part = nullptr;
    if (hipMalloc(reinterpret_cast<void**>(&part), (size_t)d.splits() * M * N * sizeof(float)) != hipSuccess)
      return fail(VLA_E_NOMEM, "gemm partials");
    g.out = part;
    hipError_t e = launch_dense(et, d, g, s);
    if (e == hipSuccess) e = launch_sum_partials(y, part, d.splits(), (size_t)M * N, s);
    hipError_t e2 = hipStreamSynchronize(s);
    hipFree(part);
    if (e != hipSuccess || e2 != hipSuccess)
      return fail(VLA_E_DEVICE, "gemm: %s", hipGetErrorString(e != hipSuccess ? e : e2));
    return VLA_OK;
  }
  DenseLaunch d = dense_launch(et, g, 1, variant);
  if (variant == 2 && !d.skinny) return fail(VLA_E_UNSUPPORTED, "shape not supported by the skinny GEMM");
  if (variant >= 3 && !d.tile) return fail(VLA_E_UNSUPPORTED, "shape not supported by the tiled GEMM");
  hipError_t e = launch_dense(et, d, g, s);
  hipError_t e2 = hipStreamSynchronize(s);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "gemm: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_attention(int32_t elem, int32_t mode, const void* q, const void* k_self, const void* v_self,
                              const void* k_cache, const void* v_cache, int32_t B, int32_t n, int32_t P, int32_t H,
                              int32_t G, int32_t hd, int32_t kv_split, void* o, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  const int causal = (mode & 4) ? 1 : 0;
  mode &= ~4;
  if (mode < 0 || mode > 2) return fail(VLA_E_ARG, "mode must be 0, 1 or 2 (+4: causal)");
  if (causal && mode == 1) return fail(VLA_E_ARG, "cross attention has no causal variant");
  if (!q || !o || (mode != 1 && (!k_self || !v_self)) || (mode != 0 && (!k_cache || !v_cache)))
    return fail(VLA_E_ARG, "NULL buffer");
  if (B < 1 || n < 1 || (mode != 0 && P < 1) || H < 1 || G < 1 || H % G) return fail(VLA_E_SHAPE, "bad shape");
  if (!(hd == 64 || hd == 128 || (elem == 1 && hd == 256))) return fail(VLA_E_UNSUPPORTED, "head_dim");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  AttnArgs a{};
  a.mode = mode; a.B = B; a.n = n; a.P = mode == 0 ? 0 : P; a.H = H; a.G = G; a.hd = hd;
  a.q = q; a.ldq = H * hd; a.ks = k_self; a.vs = v_self; a.ldkv = G * hd;
  a.kc = k_cache; a.vc = v_cache; a.o = o; a.ldo = H * hd; a.scale = 1.0f / std::sqrt((float)hd);
  a.causal = causal;
  if (H / G > 8 || H > 32) return fail(VLA_E_UNSUPPORTED, "more than 8 query heads per K/V head");
  if ((a.P + 31) / 32 + (mode == 1 ? 0 : (n + 31) / 32) > attention_max_blocks())
    return fail(VLA_E_UNSUPPORTED, "too many keys");
  const int et = elem ? ET_BF16 : ET_F32;
  if (kv_split >= 1000) {
    if (elem != 1) return fail(VLA_E_UNSUPPORTED, "the tiled attention kernel is bf16 only");
    attention_tile_split(a, kv_split - 1000);
  } else {
    attention_split(a, kv_split % 100, kv_split / 100);
  }
  void* part = nullptr;
  float* stats = nullptr;
  if (a.kv_split > 1) {
    HIP_TRY(hipMalloc(&part, attention_part_bytes(et, a)));
    HIP_TRY(hipMalloc(&stats, attention_stats_bytes(a)));
  }
  a.part = part;
  a.stats = stats;
  hipError_t e = launch_attention(et, a, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(part);
  (void)hipFree(stats);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "attention: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_adarms(int32_t elem, float* x, const float* part, int32_t nsplit, const float* alpha,
                           const float* gamma, const float* beta, int32_t M, int32_t d, float eps, void* u,
                           int32_t u_f32, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  if (!x || !gamma || !beta || !u || (nsplit > 0 && (!part || !alpha))) return fail(VLA_E_ARG, "NULL buffer");
  for (const void* q : {(const void*)x, (const void*)part, (const void*)alpha, (const void*)gamma,
                        (const void*)beta, (const void*)u})
    if (q && !al16(q)) return fail(VLA_E_ARG, "buffers must be 16-byte aligned");
  if (M < 1 || d < 4 || d % 4 || d > 4096 || nsplit < 0 || !(eps > 0.0f)) return fail(VLA_E_SHAPE, "bad shape");
  RowNormArgs a{};
  a.mode = 0; a.M = M; a.d = d; a.x = x; a.part = part; a.nsplit = nsplit; a.alpha = alpha;
  a.gamma = gamma; a.beta = beta; a.eps = eps; a.u = u; a.u_f32 = u_f32 ? 1 : 0;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_row_norm(elem, a, s);
  hipError_t e2 = hipStreamSynchronize(s);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "adarms: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_time_cond(vla_model* m, const float* t_schedule, int32_t n_steps, float* mods, float* modf,
                              void* stream) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  const vla_config& c = m->cfg;
  if (c.head_regression) return fail(VLA_E_UNSUPPORTED, "regression heads have no time input");
  if (!t_schedule || !mods || !modf || !al16(mods) || !al16(modf)) return fail(VLA_E_ARG, "bad buffer");
  if (n_steps < 1 || n_steps > VLA_MAX_STEPS) return fail(VLA_E_SHAPE, "n_steps %d not in 1..%d", n_steps, VLA_MAX_STEPS);
  for (int k = 0; k <= n_steps; ++k)
    if (!std::isfinite(t_schedule[k])) return fail(VLA_E_ARG, "schedule entry %d is not finite", k);
  const int T = n_steps, d = m->d, et = m->et;
  const size_t es = esize(et);
  const size_t modrow = (size_t)c.n_layers * 3 * m->ns * d;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  CallParams hp{};
  for (int k = 0; k <= T; ++k) hp.tau[k] = t_schedule[k];
  CallParams* cp = nullptr;
  void *e = nullptr, *h1 = nullptr, *sc = nullptr;
  hipError_t err = hipMalloc(&cp, sizeof(CallParams));
  if (err == hipSuccess) err = hipMalloc(&e, (size_t)T * d * es);
  if (err == hipSuccess) err = hipMalloc(&h1, (size_t)T * d * es);
  if (err == hipSuccess) err = hipMalloc(&sc, (size_t)T * d * es);
  if (err == hipSuccess) err = hipMemcpy(cp, &hp, sizeof(CallParams), hipMemcpyHostToDevice);
  // the same launches the plan builder records for every vla_denoise call
  if (err == hipSuccess) err = launch_time_embed(et, cp, e, T, T, d, s);
  auto gemm = [&](const void* X, const void* W, int N, const float* bias, int act, void* out, int out_f32) {
    GemmArgs g = gemm_base(m, T, N, d, X, d, W);
    g.epi = EPI_STORE; g.bias = bias; g.act = act; g.out = out; g.ldo = N; g.out_f32 = out_f32;
    return launch_dense(et, dense_launch(et, g, 1), g, s);
  };
  if (err == hipSuccess) err = gemm(e, m->W_t1, d, m->b_t1, ACT_SILU, h1, 0);
  if (err == hipSuccess) err = gemm(h1, m->W_t2, d, m->b_t2, ACT_SILU, sc, 0);
  if (err == hipSuccess) err = gemm(sc, m->W_mod, (int)modrow, m->b_mod, ACT_NONE, mods, 1);
  if (err == hipSuccess) err = gemm(sc, m->W_fm, 2 * d, m->b_fm, ACT_NONE, modf, 1);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(cp); (void)hipFree(e); (void)hipFree(h1); (void)hipFree(sc);
  if (err != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "time conditioning: %s", hipGetErrorString(err != hipSuccess ? err : e2));
  return VLA_OK;
}

vla_status vla_test_quantize_i8(const float* x, int32_t M, int32_t K, int8_t* q, float* r, void* stream) {
  if (!x || !q || !r) return fail(VLA_E_ARG, "NULL buffer");
  if (M < 1 || K < 1 || K > 16384) return fail(VLA_E_SHAPE, "bad shape");
  QuantArgs a{};
  a.M = M; a.K = K; a.x = x; a.ldx = K; a.src_type = 0; a.q = q; a.r = r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_quantize(a, s);
  hipError_t e2 = hipStreamSynchronize(s);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "quantize: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_quantize_bf16(const uint16_t* x, int32_t M, int32_t K, int32_t ldx, int8_t* q, float* r,
                                  void* stream) {
  if (!x || !q || !r) return fail(VLA_E_ARG, "NULL buffer");
  if (M < 1 || K < 1 || K > 16384 || ldx < K) return fail(VLA_E_SHAPE, "bad shape");
  QuantArgs a{};
  a.M = M; a.K = K; a.x = x; a.ldx = ldx; a.src_type = 1; a.q = q; a.r = r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_quantize(a, s);
  hipError_t e2 = hipStreamSynchronize(s);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "quantize: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_ternary_linear(const float* x, const uint8_t* w_packed, int32_t M, int32_t N, int32_t K,
                                   float scale, float* y, void* stream) {
  if (!x || !w_packed || !y || !al16(x) || !al16(w_packed) || !al16(y)) return fail(VLA_E_ARG, "bad buffer");
  if (M < 1 || N < 1 || K < 64 || K % 64 || K > 16384) return fail(VLA_E_SHAPE, "bad shape");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Tiling t = tern_tiling(M, N, K, 1);
  int8_t* q8 = nullptr;
  float *r8 = nullptr, *sc = nullptr;
  HIP_TRY(hipMalloc(&q8, (size_t)M * K));
  HIP_TRY(hipMalloc(&r8, (size_t)M * 4));
  HIP_TRY(hipMalloc(&sc, (size_t)N * 4));
  std::vector<float> hs(N, scale);
  HIP_TRY(hipMemcpy(sc, hs.data(), (size_t)N * 4, hipMemcpyHostToDevice));
  QuantArgs qa{};
  qa.M = M; qa.K = K; qa.x = x; qa.ldx = K; qa.src_type = 0; qa.q = q8; qa.r = r8;
  TernArgs a{};
  a.M = M; a.N = N; a.K = K; a.x = q8; a.w = w_packed; a.rscale = r8; a.wscale = sc;
  a.ks = t.nc * 256; a.nsplit = 1; a.n_tiles = t.n_tiles;
  a.e.M = M; a.e.N = N; a.e.K = K; a.e.epi = EPI_STORE; a.e.out = y; a.e.ldo = N; a.e.out_f32 = 1;
  hipError_t e = launch_quantize(qa, s);
  if (e == hipSuccess) e = launch_ternary_gemm(a, t.ms, t.units, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(q8); (void)hipFree(r8); (void)hipFree(sc);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "ternary linear: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_ternary_gemm(const int8_t* q, const float* r, const uint8_t* w_packed, const float* wscale,
                                 int32_t M, int32_t N, int32_t K, int32_t variant, int32_t iters, float* y,
                                 float* us_per_launch, void* stream) {
  if (!q || !r || !w_packed || !wscale || !y || !al16(q) || !al16(w_packed) || !al16(y))
    return fail(VLA_E_ARG, "bad buffer");
  if (variant < 0 || variant > 9) return fail(VLA_E_ARG, "variant must be 0 (MFMA), 1 (dot4) or 2..9 (tile)");
  if (variant >= 2 && !tern_tile_eligible(M, N, K))
    return fail(VLA_E_SHAPE, "the tiled kernel needs M >= 128 and K % 128 == 0");
  if (iters < 1 || iters > 10000) return fail(VLA_E_ARG, "iters must be 1..10000");
  if (M < 1 || N < 1 || K < 64 || K % 64 || K > 16384) return fail(VLA_E_SHAPE, "bad shape");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Tiling t = tern_tiling(M, N, K, 1);
  TernArgs a{};
  a.M = M; a.N = N; a.K = K; a.x = q; a.w = w_packed; a.rscale = r; a.wscale = wscale;
  a.ks = t.nc * 256; a.nsplit = 1; a.n_tiles = t.n_tiles;
  a.e.M = M; a.e.N = N; a.e.K = K; a.e.epi = EPI_STORE; a.e.out = y; a.e.ldo = N; a.e.out_f32 = 1;
  auto run = [&]() {
    // (row tile / 32, waves, K groups)
    static const int tile_cfg[8][3] = {{1, 4, 1}, {2, 4, 1}, {4, 4, 1}, {2, 8, 1}, {4, 8, 1}, {1, 8, 2}, {2, 8, 2},
                                       {4, 8, 2}};
    if (variant >= 2)
      return launch_ternary_tile(a, tile_cfg[variant - 2][0], tile_cfg[variant - 2][1], tile_cfg[variant - 2][2], s);
    return variant == 0 ? launch_ternary_gemm(a, t.ms, t.units, s) : launch_ternary_dot4(a, s);
  };
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = run();
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  for (int i = 0; i < iters && e == hipSuccess; ++i) e = run();
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  hipError_t e2 = hipStreamSynchronize(s);
  float ms = 0.0f;
  if (e == hipSuccess && e2 == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "ternary gemm: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  if (us_per_launch) *us_per_launch = 1000.0f * ms / (float)iters;
  return VLA_OK;
}

vla_status vla_test_rope(int32_t elem, void* x, int32_t rows, int32_t rows_per_request, int32_t ld, int32_t col0,
                         int32_t nheads, int32_t hd, int32_t pos0, float base, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  if (!x) return fail(VLA_E_ARG, "NULL buffer");
  if (rows < 1 || rows_per_request < 1 || nheads < 1 || hd < 2 || hd % 2 || col0 < 0 || pos0 < 0 ||
      col0 + nheads * hd > ld || !(base > 1.0f))
    return fail(VLA_E_SHAPE, "bad RoPE shape");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_rope(elem ? ET_BF16 : ET_F32, x, rows, rows_per_request, ld, col0, nheads, hd, pos0, base, s);
  hipError_t e2 = hipStreamSynchronize(s);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "rope: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

}  // extern "C"

// ----------------------------------------------------------------------------
// The prefix stage: a vision-language backbone's prefill (Algorithm 1's
// h = VLM-Prefix(...), one bidirectional pass over the prefix tokens; App. A.2
// items 1-2: the final-layer hidden states before the output projection are
// the cross-attention source).  A backbone layer is a self-attention sublayer
// and an MLP sublayer with pre-norms, so it is held as a vla_model of such
// layers whose static modulation table carries the norm gains as
// (gamma = g, beta = 0, alpha = 1); the prefill runs the expert's kernels at
// M = B * P token rows.

namespace {

struct PrefillPlan {
  int B = 0, P = 0;
  std::vector<void*> allocs;
  CallParams* cp = nullptr;     // a valid parameter block for the attention launches (no cache is read)
  float* x = nullptr;           // residual stream [M][d] fp32
  void* u = nullptr;            // norm output [M][d] (fp32 for W2A8 backbones)
  void *qkv = nullptr, *o = nullptr, *h = nullptr;
  float* part = nullptr;        // split-K partials of the residual projections
  void* apart = nullptr;        // attention key-split partials
  float* astats = nullptr;
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  const void* embeds = nullptr;  // this call's input rows
  void* out = nullptr;           // this call's output rows
  std::vector<Op> ops;
  ~PrefillPlan() {
    for (void* p : allocs) (void)hipFree(p);
  }
};

vla_status validate_backbone(const vla_backbone_config* c) {
  if (!c) return fail(VLA_E_ARG, "config is NULL");
  if (c->mlp < 0 || c->mlp > 3) return fail(VLA_E_ARG, "mlp %d out of range", c->mlp);
  if (c->wtype != VLA_W_BF16 && c->wtype != VLA_W_TERNARY)
    return fail(VLA_E_UNSUPPORTED, "backbone wtype must be VLA_W_BF16 or VLA_W_TERNARY");
  if (c->n_layers < 1 || c->d_model < 8 || c->n_heads < 1 || c->n_kv_heads < 1 || c->d_ff < 16)
    return fail(VLA_E_SHAPE, "non-positive dimension in backbone config");
  if (c->n_heads % c->n_kv_heads) return fail(VLA_E_SHAPE, "n_heads %% n_kv_heads != 0");
  if (!(c->head_dim == 64 || c->head_dim == 128 || c->head_dim == 256))
    return fail(VLA_E_UNSUPPORTED, "head_dim %d unsupported (64, 128, 256)", c->head_dim);
  const int m = c->wtype == VLA_W_TERNARY ? 64 : 8;
  if (c->d_model % m || (c->n_heads * c->head_dim) % m || c->d_ff % (m > 16 ? m : 16))
    return fail(VLA_E_SHAPE, "d_model and H*hd must be multiples of %d, d_ff of %d", m, m > 16 ? m : 16);
  if (c->d_model > 4096) return fail(VLA_E_UNSUPPORTED, "d_model > 4096");
  if (c->n_heads / c->n_kv_heads > 8 || c->n_heads > 32)
    return fail(VLA_E_UNSUPPORTED, "more than 8 query heads per K/V head or more than 32 heads");
  if (c->d_ff > 65536) return fail(VLA_E_UNSUPPORTED, "d_ff > 65536");
  if (!std::isfinite(c->rope_base) || (c->rope_base != 0.0f && !(c->rope_base > 1.0f)))
    return fail(VLA_E_ARG, "rope_base must be 0 or > 1");
  if (!(c->rms_eps > 0.0f) || !std::isfinite(c->rms_eps)) return fail(VLA_E_ARG, "rms_eps must be finite and > 0");
  return VLA_OK;
}

int backbone_weight_count(const vla_backbone_config& c) {
  const int mats = 4 + (c.mlp == VLA_MLP_GELU ? 2 : 3);
  return 1 + c.n_layers * (2 + mats * (c.wtype == VLA_W_TERNARY ? 2 : 1));
}

}  // namespace

struct vla_backbone {
  vla_backbone_config cfg{};
  std::unique_ptr<vla_model> m;
  std::map<std::pair<int, int>, std::unique_ptr<PrefillPlan>> plans;
  ~vla_backbone() {
    plans.clear();
    m.reset();
  }
};

namespace {

vla_status backbone_create_impl(const vla_backbone_config* bc, const void* const* weights, int32_t n_weights,
                                vla_backbone** out) {
  std::unique_ptr<vla_backbone> bb(new vla_backbone());
  bb->cfg = *bc;
  bb->m.reset(new vla_model());
  vla_model* m = bb->m.get();
  vla_config& c = m->cfg;
  c.n_layers = bc->n_layers;
  c.d_model = bc->d_model;
  c.n_heads = bc->n_heads;
  c.head_dim = bc->head_dim;
  c.n_kv_heads = bc->n_kv_heads;
  c.d_ff = bc->d_ff;
  c.mlp = bc->mlp;
  c.wtype = bc->wtype;
  c.rms_eps = bc->rms_eps;
  c.head_regression = 1;      // static modulation, no time input
  m->tern = bc->wtype == VLA_W_TERNARY;
  m->et = ET_BF16;
  m->d = bc->d_model;
  m->dq = bc->n_heads * bc->head_dim;
  m->dkv = bc->n_kv_heads * bc->head_dim;
  m->ns = 2;
  const int d = m->d, F = bc->d_ff, L = bc->n_layers, dq = m->dq, dkv = m->dkv;
  TableReader tr{weights, n_weights};
  const void* p;
  // norm gains as the static modulation table [L][2][3][d] = (g, 0, 1) per
  // sublayer, the final one as [2][d] = (g_f, 0)
  std::vector<float> tab((size_t)L * 2 * 3 * d, 0.0f), fin((size_t)2 * d, 0.0f);
  auto gain = [&](const char* what, float* dst) -> vla_status {
    VLA_TRY(tr.next(&p, what));
    HIP_TRY(hipMemcpy(dst, p, (size_t)d * 4, hipMemcpyDeviceToHost));
    for (int i = 0; i < d; ++i)
      if (!std::isfinite(dst[i])) return fail(VLA_E_ARG, "norm gain %s is not finite", what);
    return VLA_OK;
  };
  auto mat = [&](const char* what, const void** src, float* scale) -> vla_status {
    VLA_TRY(tr.next(src, what));
    *scale = 1.0f;
    if (!m->tern) return VLA_OK;
    const void* sp;
    VLA_TRY(tr.next(&sp, "ternary scale"));
    vla_status st = VLA_OK;
    *scale = read_scale(sp, &st);
    return st;
  };
  VLA_TRY(gain("g_f", fin.data()));
  m->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    float* row = tab.data() + (size_t)l * 2 * 3 * d;
    VLA_TRY(gain("g_att", row));
    for (int i = 0; i < d; ++i) row[2 * d + i] = 1.0f;
    SubW at;
    at.kind = K_SELF;
    const void *wq, *wk, *wv, *wo;
    float sq, sk, sv, so;
    VLA_TRY(mat("W_q", &wq, &sq));
    VLA_TRY(mat("W_k", &wk, &sk));
    VLA_TRY(mat("W_v", &wv, &sv));
    VLA_TRY(mat("W_o", &wo, &so));
    at.n_qkv = dq + 2 * dkv;
    VLA_TRY(fuse(m, &at.qkv, &at.s_qkv, {{wq, dq, sq}, {wk, dkv, sk}, {wv, dkv, sv}}, d, false));
    VLA_TRY(fuse(m, &at.o, &at.s_o, {{wo, d, so}}, dq, false));
    VLA_TRY(gain("g_mlp", row + 3 * d));
    for (int i = 0; i < d; ++i) row[5 * d + i] = 1.0f;
    SubW ml;
    ml.kind = K_MLP;
    if (bc->mlp == VLA_MLP_GELU) {
      const void *w1, *w2;
      float s1, s2;
      VLA_TRY(mat("W1", &w1, &s1));
      VLA_TRY(mat("W2", &w2, &s2));
      VLA_TRY(fuse(m, &ml.gu, &ml.s_gu, {{w1, F, s1}}, d, false));
      VLA_TRY(fuse(m, &ml.dn, &ml.s_dn, {{w2, d, s2}}, F, false));
    } else {
      const void *wg, *wu, *wd;
      float sg, su, sd;
      VLA_TRY(mat("W_g", &wg, &sg));
      VLA_TRY(mat("W_u", &wu, &su));
      VLA_TRY(mat("W_d", &wd, &sd));
      VLA_TRY(fuse(m, &ml.gu, &ml.s_gu, {{wg, F, sg}, {wu, F, su}}, d, true));
      VLA_TRY(fuse(m, &ml.dn, &ml.s_dn, {{wd, d, sd}}, F, false));
    }
    m->layers[l] = {at, ml};
  }
  if (tr.i != n_weights) return fail(VLA_E_ARG, "weight table has %d entries, expected %d", n_weights, tr.i);
  Alloc al{m->allocs};
  VLA_TRY(al((void**)&m->mod_static, tab.size() * 4));
  HIP_TRY(hipMemcpy(m->mod_static, tab.data(), tab.size() * 4, hipMemcpyHostToDevice));
  VLA_TRY(al((void**)&m->modf_static, fin.size() * 4));
  HIP_TRY(hipMemcpy(m->modf_static, fin.data(), fin.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipDeviceSynchronize());
  *out = bb.release();
  return VLA_OK;
}

vla_status build_prefill_plan(vla_backbone* bb, PrefillPlan* p) {
  vla_model* m = bb->m.get();
  const vla_backbone_config& bc = bb->cfg;
  const int B = p->B, P = p->P, M = B * P, d = m->d, dq = m->dq, dkv = m->dkv, F = bc.d_ff, L = bc.n_layers;
  const int H = bc.n_heads, G = bc.n_kv_heads, hd = bc.head_dim, nqkv = dq + 2 * dkv;
  const int et = m->et;
  const size_t es = esize(et);
  const bool tern = m->tern;
  const bool glu = bc.mlp != VLA_MLP_GELU;
  Alloc al{p->allocs};
  VLA_TRY(al((void**)&p->cp, sizeof(CallParams)));
  HIP_TRY(hipMemset(p->cp, 0, sizeof(CallParams)));
  VLA_TRY(al((void**)&p->x, (size_t)M * d * 4));
  VLA_TRY(al(&p->u, (size_t)M * d * (tern ? 4 : es)));
  VLA_TRY(al(&p->qkv, (size_t)M * nqkv * es));
  VLA_TRY(al(&p->o, (size_t)M * dq * es));
  VLA_TRY(al(&p->h, (size_t)M * F * (tern ? 4 : es)));
  if (tern) {
    VLA_TRY(al((void**)&p->q8, (size_t)M * std::max(std::max(d, dq), F)));
    VLA_TRY(al((void**)&p->r8, (size_t)M * 4));
  }
  Builder bld{m, &p->ops, &p->apart, &p->astats};
  const size_t modrow = (size_t)2 * 3 * d;
  auto gam = [&](int l, int j) { return m->mod_static + (size_t)l * modrow + (size_t)j * 3 * d; };
  size_t part_need = 0;
  PrefillPlan* pp = p;
  float** partp = &p->part;

  {  // the residual stream starts as the input rows; first norm
    RowNormArgs r{};
    r.mode = 2; r.M = M; r.d = d; r.x = p->x; r.gamma = gam(0, 0); r.beta = gam(0, 0) + d; r.eps = bc.rms_eps;
    r.u = p->u; r.u_f32 = tern ? 1 : 0;
    if (tern) {
      r.q = p->q8;
      r.qr = p->r8;
    }
    bld.ops->push_back(Op{[=](hipStream_t s) {
                            RowNormArgs q = r;
                            q.x_in = pp->embeds;
                            return launch_row_norm(et, q, s);
                          },
                          op_info(VLA_OP_SMALL, M, d, 0, (double)M * d * (es + 4.0 + (tern ? 5.0 : es)), 0.0)});
  }
  // residual projection of a dense backbone: split-K partials summed by the
  // following row kernel, or the residual update in the GEMM's epilogue
  auto resid_gemm = [&](GemmArgs g, const float* alp, RowNormArgs& rn) {
    g.epi = EPI_PARTIAL;
    const DenseLaunch dl = dense_launch(et, g, 1);
    if (dl.skinny || (dl.tile && dl.tl.nsplit > 1)) {
      g.out = nullptr;
      g.ldo = d;
      part_need = std::max(part_need, (size_t)dl.splits() * M * d);
      const GemmArgs gg = g;
      const double bytes = (double)g.N * g.K * es + (double)g.M * g.K * es + 4.0 * dl.splits() * g.M * g.N;
      bld.ops->push_back(Op{[=](hipStream_t s) {
                              GemmArgs q = gg;
                              q.out = *partp;
                              return launch_dense(et, dl, q, s);
                            },
                            op_info(VLA_OP_GEMM, g.M, g.N, g.K, bytes, 2.0 * g.M * g.N * g.K)});
      rn.nsplit = dl.splits();
      rn.alpha = alp;
    } else {
      g.epi = EPI_RESID;
      g.xres = p->x;
      g.ldxr = d;
      g.alpha = alp;
      bld.gemm(g, 1);
      rn.nsplit = 0;
      rn.alpha = nullptr;
    }
  };
  auto tern_resid = [&](const SubW& sw, const void* W, const float* ws, int K, const float* alp) {
    TernArgs t{};
    t.M = M; t.N = d; t.K = K; t.x = p->q8; t.w = (const uint8_t*)W; t.rscale = p->r8; t.wscale = ws;
    t.e = gemm_base(m, M, d, K, nullptr, 0, nullptr);
    t.e.epi = EPI_RESID;
    t.e.xres = p->x;
    t.e.ldxr = d;
    t.e.alpha = alp;
    bld.tern(t, 1);
    (void)sw;
  };
  // row kernel finishing a residual update and normalising for what follows;
  // after the last layer it writes the final norm into the call's output
  auto norm_op = [&](RowNormArgs nr, bool final_out) {
    const double bytes = (double)M * d * (8.0 + 4.0 * std::min(nr.nsplit, 1) + (nr.u_f32 ? 4.0 : es));
    bld.ops->push_back(Op{[=](hipStream_t s) {
                            RowNormArgs r = nr;
                            r.part = *partp;
                            if (final_out) r.u = pp->out;
                            return launch_row_norm(et, r, s);
                          },
                          op_info(VLA_OP_SMALL, M, d, nr.nsplit, bytes, 0.0)});
  };

  for (int l = 0; l < L; ++l) {
    const SubW& at = m->layers[l][0];
    const SubW& ml = m->layers[l][1];
    // ---- attention sublayer: [q | k | v] = u W^T, RoPE, bidirectional attention, W_o
    if (!tern) {
      GemmArgs g = gemm_base(m, M, nqkv, d, p->u, d, at.qkv);
      g.epi = EPI_STORE;
      g.out = p->qkv;
      g.ldo = nqkv;
      bld.gemm(g, 1);
    } else {
      TernArgs t{};
      t.M = M; t.N = nqkv; t.K = d; t.x = p->q8; t.w = (const uint8_t*)at.qkv; t.rscale = p->r8; t.wscale = at.s_qkv;
      t.e = gemm_base(m, M, nqkv, d, nullptr, 0, nullptr);
      t.e.epi = EPI_STORE;
      t.e.out = p->qkv;
      t.e.ldo = nqkv;
      bld.tern(t, 1);
    }
    if (bc.rope_base > 0.0f) {
      void* qkvp = p->qkv;
      const float base = bc.rope_base;
      bld.small([=](hipStream_t s) {
        hipError_t e = launch_rope(et, qkvp, M, P, nqkv, 0, H, hd, 0, base, s);
        return e != hipSuccess ? e : launch_rope(et, qkvp, M, P, nqkv, dq, G, hd, 0, base, s);
      }, M, dq + dkv, 0, 2.0 * M * (dq + dkv) * es);
    }
    AttnArgs a{};
    a.mode = 0;
    a.causal = 0;
    a.B = B; a.n = P; a.P = 0; a.H = H; a.G = G; a.hd = hd;
    a.q = p->qkv; a.ldq = nqkv;
    a.ks = (const char*)p->qkv + (size_t)dq * es;
    a.vs = (const char*)p->qkv + (size_t)(dq + dkv) * es;
    a.ldkv = nqkv;
    a.kc = nullptr;
    a.vc = nullptr;
    a.cp = p->cp;
    a.layer_off = 0;
    a.o = p->o;
    a.ldo = dq;
    a.scale = 1.0f / std::sqrt((float)hd);
    bld.attn(a);
    RowNormArgs nr{};
    nr.mode = 0; nr.M = M; nr.d = d; nr.x = p->x; nr.eps = bc.rms_eps; nr.u = p->u; nr.u_f32 = tern ? 1 : 0;
    nr.gamma = gam(l, 1);
    nr.beta = gam(l, 1) + d;
    if (tern) {
      nr.q = p->q8;
      nr.qr = p->r8;
    }
    if (!tern) {
      resid_gemm(gemm_base(m, M, d, dq, p->o, dq, at.o), gam(l, 0) + 2 * d, nr);
    } else {
      QuantArgs q{};
      q.M = M; q.K = dq; q.x = p->o; q.ldx = dq; q.src_type = 1; q.q = p->q8; q.r = p->r8;
      bld.quant(q);
      tern_resid(at, at.o, at.s_o, dq, gam(l, 0) + 2 * d);
    }
    norm_op(nr, false);
    // ---- MLP sublayer
    const bool last = l == L - 1;
    RowNormArgs nm{};
    nm.mode = 0; nm.M = M; nm.d = d; nm.x = p->x; nm.eps = bc.rms_eps;
    if (!last) {
      nm.gamma = gam(l + 1, 0);
      nm.beta = gam(l + 1, 0) + d;
      nm.u = p->u;
      nm.u_f32 = tern ? 1 : 0;
      if (tern) {
        nm.q = p->q8;
        nm.qr = p->r8;
      }
    } else {   // final norm, written as the element type into the call's output
      nm.gamma = m->modf_static;
      nm.beta = m->modf_static + d;
      nm.u_f32 = 0;
    }
    const int ngu = glu ? 2 * F : F;
    if (!tern) {
      GemmArgs g = gemm_base(m, M, ngu, d, p->u, d, ml.gu);
      g.epi = glu ? EPI_GLU : EPI_STORE;
      g.act = mlp_act(bc.mlp);
      g.out = p->h;
      g.ldo = F;
      bld.gemm(g, glu ? 2 : 1);
      resid_gemm(gemm_base(m, M, d, F, p->h, F, ml.dn), gam(l, 1) + 2 * d, nm);
    } else {
      TernArgs t{};
      t.M = M; t.N = ngu; t.K = d; t.x = p->q8; t.w = (const uint8_t*)ml.gu; t.rscale = p->r8; t.wscale = ml.s_gu;
      t.e = gemm_base(m, M, ngu, d, nullptr, 0, nullptr);
      t.e.epi = glu ? EPI_GLU : EPI_STORE;
      t.e.act = mlp_act(bc.mlp);
      t.e.out = p->h;
      t.e.ldo = F;
      t.e.out_f32 = 1;
      bld.tern(t, glu ? 2 : 1);
      QuantArgs q{};
      q.M = M; q.K = F; q.x = p->h; q.ldx = F; q.src_type = 0; q.q = p->q8; q.r = p->r8;
      bld.quant(q);
      tern_resid(ml, ml.dn, ml.s_dn, F, gam(l, 1) + 2 * d);
    }
    norm_op(nm, last);
  }
  if (part_need) VLA_TRY(al((void**)&p->part, part_need * 4));
  if (bld.part_need) VLA_TRY(al(&p->apart, bld.part_need));
  if (bld.stats_need) VLA_TRY(al((void**)&p->astats, bld.stats_need));
  HIP_TRY(hipDeviceSynchronize());
  return VLA_OK;
}

}  // namespace

extern "C" {

int32_t vla_backbone_weight_count(const vla_backbone_config* cfg) {
  if (!cfg || validate_backbone(cfg) != VLA_OK) return -1;
  return backbone_weight_count(*cfg);
}

vla_status vla_backbone_create(const vla_backbone_config* cfg, const void* const* weights, int32_t n_weights,
                               vla_backbone** out) {
  if (!out) return fail(VLA_E_ARG, "out is NULL");
  *out = nullptr;
  VLA_TRY(validate_backbone(cfg));
  if (!weights) return fail(VLA_E_ARG, "weight table is NULL");
  const int want = backbone_weight_count(*cfg);
  if (n_weights != want) return fail(VLA_E_ARG, "weight table has %d entries, expected %d", n_weights, want);
  for (int i = 0; i < n_weights; ++i) {
    if (!weights[i]) return fail(VLA_E_ARG, "weight entry %d is NULL", i);
    if (!al16(weights[i])) return fail(VLA_E_ARG, "weight entry %d is not 16-byte aligned", i);
  }
  return backbone_create_impl(cfg, weights, n_weights, out);
}

void vla_backbone_destroy(vla_backbone* bb) { delete bb; }

vla_status vla_prefix_prefill(vla_backbone* bb, const void* embeds, int32_t batch, int32_t prefix_len,
                              void* hidden_out, void* stream) {
  if (!bb) return fail(VLA_E_ARG, "backbone is NULL");
  if (!embeds || !hidden_out) return fail(VLA_E_ARG, "embeds / hidden_out is NULL");
  if (!al16(embeds) || !al16(hidden_out)) return fail(VLA_E_ARG, "buffers must be 16-byte aligned");
  if (batch < 1 || prefix_len < 1) return fail(VLA_E_SHAPE, "batch and prefix_len must be >= 1");
  if ((long long)batch * prefix_len > 65536) return fail(VLA_E_UNSUPPORTED, "batch * prefix_len > 65536");
  if ((prefix_len + 31) / 32 > attention_max_blocks())
    return fail(VLA_E_UNSUPPORTED, "prefix_len beyond %d rows", 32 * attention_max_blocks());
  auto key = std::make_pair((int)batch, (int)prefix_len);
  auto it = bb->plans.find(key);
  PrefillPlan* p;
  if (it == bb->plans.end()) {
    if (bb->plans.size() >= 4) bb->plans.erase(bb->plans.begin());
    std::unique_ptr<PrefillPlan> np(new PrefillPlan());
    np->B = batch;
    np->P = prefix_len;
    VLA_TRY(build_prefill_plan(bb, np.get()));
    p = np.get();
    bb->plans[key] = std::move(np);
  } else {
    p = it->second.get();
  }
  p->embeds = embeds;
  p->out = hidden_out;
  VLA_TRY(run_ops(p->ops, reinterpret_cast<hipStream_t>(stream)));
  return VLA_OK;
}

}  // extern "C"

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
  if (c->pattern < 0 || c->pattern > 2) return fail(VLA_E_ARG, "pattern %d out of range", c->pattern);
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
  float *b_in = nullptr, *b_s = nullptr, *b_out = nullptr;
  void *W_t1 = nullptr, *W_t2 = nullptr, *W_fm = nullptr, *W_mod = nullptr;
  float *b_t1 = nullptr, *b_t2 = nullptr, *b_fm = nullptr, *b_mod = nullptr;
  float *mod_static = nullptr, *modf_static = nullptr;
  std::vector<std::vector<SubW>> layers;
  std::map<std::tuple<int, int, int>, std::unique_ptr<Plan>> plans;
  std::map<std::pair<int, int>, std::unique_ptr<PrefixWs>> prefix_ws;
  int loop_mode = 1;
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

using Op = std::function<hipError_t(hipStream_t)>;

struct Plan {
  int B = 0, P = 0, T = 0;
  std::vector<void*> allocs;
  CallParams* cp = nullptr;
  float *a = nullptr, *xs = nullptr, *x = nullptr, *rowss = nullptr, *mods = nullptr, *modf = nullptr;
  void *e = nullptr, *h1 = nullptr, *sc = nullptr, *qkv = nullptr, *o = nullptr, *h = nullptr;
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  float* ws = nullptr;
  unsigned* cnt = nullptr;
  size_t ws_floats = 0, n_cnt = 0;
  std::vector<Op> ops;
  hipGraphExec_t exec = nullptr;
  ~Plan() {
    if (exec) (void)hipGraphExecDestroy(exec);
    for (void* p : allocs) (void)hipFree(p);
  }
};

struct PrefixWs {
  std::vector<void*> allocs;
  float* ws = nullptr;
  unsigned* cnt = nullptr;
  size_t ws_floats = 0, n_cnt = 0;
  int8_t* q8 = nullptr;
  float* r8 = nullptr;
  ~PrefixWs() {
    for (void* p : allocs) (void)hipFree(p);
  }
};

struct Tiling {
  int ms, nsub, nc, nsplit, n_tiles, m_tiles, units;
};

Tiling gemm_tiling(int et, int M, int N, int K, int nsub, int force_nsplit = 0) {
  Tiling t{};
  t.ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  t.nsub = nsub;
  t.m_tiles = cdiv(M, 16 * t.ms);
  t.n_tiles = cdiv(N, 64 * nsub);
  const int KC = gemm_chunk_k(et);
  const int base = t.m_tiles * t.n_tiles;
  t.nc = 1;
  for (int nc : {4, 2, 1}) {
    const int nsplit = cdiv(K, nc * KC);
    // Largest K-slice that still yields one workgroup per CU (or the split
    // count a test asks for).
    const bool ok = force_nsplit > 0 ? nsplit >= force_nsplit : base * nsplit >= 256;
    if (ok) {
      t.nc = nc;
      break;
    }
  }
  t.nsplit = cdiv(K, t.nc * KC);
  t.units = base * t.nsplit;
  return t;
}

Tiling tern_tiling(int M, int N, int K, int nsub) {
  Tiling t{};
  t.ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  t.nsub = nsub;
  t.m_tiles = cdiv(M, 16 * t.ms);
  t.n_tiles = cdiv(N, 64 * nsub);
  const int base = t.m_tiles * t.n_tiles;
  for (int nc : {8, 4, 2, 1}) {
    const int nsplit = cdiv(K, nc * 256);
    if (base * nsplit >= 256 || nc == 1) {
      t.nc = nc;
      t.nsplit = nsplit;
      break;
    }
  }
  t.units = base * t.nsplit;
  return t;
}

// Collects the launches of a plan and the workspace they need.
struct Builder {
  vla_model* m;
  std::vector<Op>* ops;
  float** ws;
  unsigned** cnt;
  size_t ws_need = 0, cnt_need = 0;

  void gemm(GemmArgs a, int nsub, int force_nsplit = 0) {
    const int et = m->et;
    const Tiling t = gemm_tiling(et, a.M, a.N, a.K, nsub, force_nsplit);
    a.ks = t.nc * gemm_chunk_k(et);
    a.nsplit = t.nsplit;
    a.n_tiles = t.n_tiles;
    if (t.nsplit > 1) {
      ws_need = std::max(ws_need, (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, nsub));
      cnt_need = std::max(cnt_need, (size_t)t.m_tiles * t.n_tiles);
    }
    float** wsp = ws;
    unsigned** cntp = cnt;
    ops->push_back([=](hipStream_t s) {
      GemmArgs g = a;
      g.ws = *wsp;
      g.cnt = *cntp;
      return launch_gemm(et, t.ms, nsub, t.nc, g, t.units, s);
    });
  }

  void tern(TernArgs a, int nsub) {
    const Tiling t = tern_tiling(a.M, a.N, a.K, nsub);
    a.ks = t.nc * 256;
    a.nsplit = t.nsplit;
    a.n_tiles = t.n_tiles;
    if (t.nsplit > 1) {
      ws_need = std::max(ws_need, (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, nsub));
      cnt_need = std::max(cnt_need, (size_t)t.m_tiles * t.n_tiles);
    }
    float** wsp = ws;
    unsigned** cntp = cnt;
    ops->push_back([=](hipStream_t s) {
      TernArgs g = a;
      g.ws = reinterpret_cast<int*>(*wsp);
      g.cnt = *cntp;
      return launch_ternary_gemm(g, t.ms, t.units, s);
    });
  }

  void attn(AttnArgs a) {
    const int QT = cdiv(a.n, 16);
    const int total = (a.mode == 0 ? 0 : a.P) + (a.mode == 1 ? 0 : a.n);
    const int base = a.B * a.H * QT;
    int split = std::max(1, std::min(cdiv(256, base), cdiv(total, 32)));
    a.key_chunk = cdiv(cdiv(total, split), 32) * 32;
    a.kv_split = cdiv(total, a.key_chunk);
    if (a.kv_split > 1) {
      ws_need = std::max(ws_need, attention_ws_floats(a));
      cnt_need = std::max(cnt_need, (size_t)base);
    }
    const int et = m->et;
    float** wsp = ws;
    unsigned** cntp = cnt;
    ops->push_back([=](hipStream_t s) {
      AttnArgs g = a;
      g.ws = *wsp;
      g.cnt = *cntp;
      return launch_attention(et, g, s);
    });
  }

  void quant(QuantArgs q) {
    ops->push_back([=](hipStream_t s) { return launch_quantize(q, s); });
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
  a.eps = m->cfg.rms_eps;
  return a;
}

void set_adarms(GemmArgs& a, const float* rowss, int np, const float* gamma, const float* beta) {
  a.rowss = rowss;
  a.rowss_np = np;
  a.gamma = gamma;
  a.beta = beta;
}

int mlp_act(int mlp) {
  switch (mlp) {
    case VLA_MLP_GELU:
    case VLA_MLP_GEGLU: return ACT_GELU;
    case VLA_MLP_SWIGLU: return ACT_SILU;
    default: return ACT_RELU2;
  }
}

vla_status build_plan(vla_model* m, Plan* p) {
  const vla_config& c = m->cfg;
  const int B = p->B, P = p->P, T = p->T;
  const int n = c.n_action, A = c.d_action, S = c.d_state, d = m->d, F = c.d_ff;
  const int M = B * n, L = c.n_layers, ns = m->ns, dq = m->dq, dkv = m->dkv, hd = c.head_dim;
  const int et = m->et;
  const size_t es = esize(et);
  const int np = cdiv(d, 64);
  const size_t modrow = (size_t)L * 3 * ns * d;
  Alloc al{p->allocs};
  VLA_TRY(al((void**)&p->cp, sizeof(CallParams)));
  VLA_TRY(al((void**)&p->a, (size_t)M * A * 4));
  VLA_TRY(al((void**)&p->xs, (size_t)B * d * 4));
  VLA_TRY(al((void**)&p->x, (size_t)M * d * 4));
  VLA_TRY(al((void**)&p->rowss, (size_t)np * M * 4));
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

  Builder bld{m, &p->ops, &p->ws, &p->cnt};
  std::vector<Op>& ops = p->ops;
  CallParams* cp = p->cp;

  ops.push_back([=](hipStream_t s) {
    return launch_init_chunk(et, cp, p->a, p->xs, m->W_s, m->b_s, m->b_in, B, n, A, S, d, s);
  });
  if (!c.head_regression) {
    ops.push_back([=](hipStream_t s) { return launch_time_embed(et, cp, p->e, T, T, d, s); });
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

  const size_t layer_block = (size_t)2 * B * c.n_kv_heads * P * hd;  // elements per cache layer
  for (int k = 0; k < T; ++k) {
    const float* modk = c.head_regression ? m->mod_static : p->mods + (size_t)k * modrow;
    const float* modfk = c.head_regression ? m->modf_static : p->modf + (size_t)k * 2 * d;
    ops.push_back([=](hipStream_t s) {
      return launch_embed(et, p->a, m->W_in, p->xs, m->E_pos, p->x, p->rowss, B, n, A, d, s);
    });
    for (int l = 0; l < L; ++l) {
      const std::vector<SubW>& subs = m->layers[l];
      for (int j = 0; j < (int)subs.size(); ++j) {
        const SubW& sw = subs[j];
        const float* gam = modk + ((size_t)l * ns + j) * 3 * d;
        const float* bet = gam + d;
        const float* alp = gam + 2 * d;
        if (sw.kind == K_MLP) {
          const bool glu = c.mlp != VLA_MLP_GELU;
          const int ngu = glu ? 2 * F : F;
          if (!m->tern) {
            GemmArgs g = gemm_base(m, M, ngu, d, p->x, d, sw.gu);
            set_adarms(g, p->rowss, np, gam, bet);
            g.epi = glu ? EPI_GLU : EPI_STORE;
            g.act = mlp_act(c.mlp);
            g.out = p->h;
            g.ldo = F;
            bld.gemm(g, glu ? 2 : 1);
            g = gemm_base(m, M, d, F, p->h, F, sw.dn);
            g.epi = EPI_RESID;
            g.xres = p->x;
            g.ldxr = d;
            g.alpha = alp;
            g.rowss_out = p->rowss;
            bld.gemm(g, 1);
          } else {
            QuantArgs q{};
            q.M = M; q.K = d; q.x = p->x; q.ldx = d; q.src_type = 0; q.adarms = 1;
            q.rowss = p->rowss; q.rowss_np = np; q.gamma = gam; q.beta = bet; q.eps = c.rms_eps;
            q.q = p->q8; q.r = p->r8;
            bld.quant(q);
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
            q.M = M; q.K = F; q.x = p->h; q.ldx = F; q.src_type = 0; q.adarms = 0; q.q = p->q8; q.r = p->r8;
            bld.quant(q);
            t = TernArgs{};
            t.M = M; t.N = d; t.K = F; t.x = p->q8; t.w = (const uint8_t*)sw.dn; t.rscale = p->r8; t.wscale = sw.s_dn;
            t.e = gemm_base(m, M, d, F, nullptr, 0, nullptr);
            t.e.epi = EPI_RESID;
            t.e.xres = p->x;
            t.e.ldxr = d;
            t.e.alpha = alp;
            t.e.rowss_out = p->rowss;
            bld.tern(t, 1);
          }
        } else {
          // Q (and self K, V) projection
          if (!m->tern) {
            GemmArgs g = gemm_base(m, M, sw.n_qkv, d, p->x, d, sw.qkv);
            set_adarms(g, p->rowss, np, gam, bet);
            g.epi = EPI_STORE;
            g.out = p->qkv;
            g.ldo = ldqkv;
            bld.gemm(g, 1);
          } else {
            QuantArgs q{};
            q.M = M; q.K = d; q.x = p->x; q.ldx = d; q.src_type = 0; q.adarms = 1;
            q.rowss = p->rowss; q.rowss_np = np; q.gamma = gam; q.beta = bet; q.eps = c.rms_eps;
            q.q = p->q8; q.r = p->r8;
            bld.quant(q);
            TernArgs t{};
            t.M = M; t.N = sw.n_qkv; t.K = d; t.x = p->q8; t.w = (const uint8_t*)sw.qkv; t.rscale = p->r8;
            t.wscale = sw.s_qkv;
            t.e = gemm_base(m, M, sw.n_qkv, d, nullptr, 0, nullptr);
            t.e.epi = EPI_STORE;
            t.e.out = p->qkv;
            t.e.ldo = ldqkv;
            bld.tern(t, 1);
          }
          AttnArgs at{};
          at.mode = sw.kind == K_SELF ? 0 : (sw.kind == K_CROSS ? 1 : 2);
          at.B = B; at.n = n; at.P = P; at.H = c.n_heads; at.G = c.n_kv_heads; at.hd = hd;
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
            GemmArgs g = gemm_base(m, M, d, dq, p->o, dq, sw.o);
            g.epi = EPI_RESID;
            g.xres = p->x;
            g.ldxr = d;
            g.alpha = alp;
            g.rowss_out = p->rowss;
            bld.gemm(g, 1);
          } else {
            QuantArgs q{};
            q.M = M; q.K = dq; q.x = p->o; q.ldx = dq; q.src_type = 1; q.adarms = 0; q.q = p->q8; q.r = p->r8;
            bld.quant(q);
            TernArgs t{};
            t.M = M; t.N = d; t.K = dq; t.x = p->q8; t.w = (const uint8_t*)sw.o; t.rscale = p->r8; t.wscale = sw.s_o;
            t.e = gemm_base(m, M, d, dq, nullptr, 0, nullptr);
            t.e.epi = EPI_RESID;
            t.e.xres = p->x;
            t.e.ldxr = d;
            t.e.alpha = alp;
            t.e.rowss_out = p->rowss;
            bld.tern(t, 1);
          }
        }
      }
    }
    // head: final adaRMS, out-projection and the Euler update
    GemmArgs g = gemm_base(m, M, A, d, p->x, d, m->W_out);
    set_adarms(g, p->rowss, np, modfk, modfk + d);
    g.epi = EPI_EULER;
    g.bias = m->b_out;
    g.a = p->a;
    g.cp = cp;
    g.step = k;
    g.regression = c.head_regression;
    g.last = (k == T - 1);
    bld.gemm(g, 1);
  }

  if (bld.ws_need) VLA_TRY(al((void**)&p->ws, bld.ws_need * 4));
  if (bld.cnt_need) {
    VLA_TRY(al((void**)&p->cnt, bld.cnt_need * 4));
    HIP_TRY(hipMemset(p->cnt, 0, bld.cnt_need * 4));
  }
  p->ws_floats = bld.ws_need;
  p->n_cnt = bld.cnt_need;
  HIP_TRY(hipDeviceSynchronize());
  return VLA_OK;
}

vla_status run_ops(const std::vector<Op>& ops, hipStream_t s) {
  for (const Op& op : ops) HIP_TRY(op(s));
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
    if (value < 0 || value > 1) return fail(VLA_E_ARG, "loop mode %d out of range", value);
    m->loop_mode = value;
    return VLA_OK;
  }
  return fail(VLA_E_ARG, "unknown option %d", option);
}

void vla_model_destroy(vla_model* m) { delete m; }

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
  const int M = B * P;
  size_t ws_need = 0, cnt_need = 0;
  const int N = 2 * m->dkv, K = m->cfg.d_prefix;
  if (m->tern) {
    const Tiling t = tern_tiling(M, N, K, 1);
    if (t.nsplit > 1) {
      ws_need = (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, 1);
      cnt_need = (size_t)t.m_tiles * t.n_tiles;
    }
  } else {
    const Tiling t = gemm_tiling(m->et, M, N, K, 1);
    if (t.nsplit > 1) {
      ws_need = (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, 1);
      cnt_need = (size_t)t.m_tiles * t.n_tiles;
    }
  }
  Alloc al{w->allocs};
  if (ws_need) VLA_TRY(al((void**)&w->ws, ws_need * 4));
  if (cnt_need) {
    VLA_TRY(al((void**)&w->cnt, cnt_need * 4));
    HIP_TRY(hipMemset(w->cnt, 0, cnt_need * 4));
  }
  if (m->tern) {
    VLA_TRY(al((void**)&w->q8, (size_t)M * K));
    VLA_TRY(al((void**)&w->r8, (size_t)M * 4));
  }
  HIP_TRY(hipDeviceSynchronize());
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

vla_status vla_prefix_kv_build(vla_model* m, const void* prefix_hidden, int32_t batch, int32_t prefix_len,
                               void* kv_cache, size_t kv_cache_bytes, void* stream) {
  if (!m) return fail(VLA_E_ARG, "model is NULL");
  if (!prefix_hidden || !kv_cache) return fail(VLA_E_ARG, "prefix_hidden / kv_cache is NULL");
  if (!al16(prefix_hidden) || !al16(kv_cache)) return fail(VLA_E_ARG, "buffers must be 16-byte aligned");
  if (batch < 1 || prefix_len < 1) return fail(VLA_E_SHAPE, "batch and prefix_len must be >= 1");
  if ((long long)batch * prefix_len > (1LL << 24)) return fail(VLA_E_UNSUPPORTED, "batch * prefix_len too large");
  if (kv_cache_bytes != vla_kv_cache_bytes(m, batch, prefix_len))
    return fail(VLA_E_SHAPE, "kv_cache_bytes %zu != %zu for batch %d, prefix_len %d", kv_cache_bytes,
                vla_kv_cache_bytes(m, batch, prefix_len), batch, prefix_len);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  PrefixWs* w = nullptr;
  VLA_TRY(get_prefix_ws(m, batch, prefix_len, &w));
  const int M = batch * prefix_len, N = 2 * m->dkv, K = m->cfg.d_prefix, hd = m->cfg.head_dim;
  const size_t layer_block = (size_t)2 * batch * m->cfg.n_kv_heads * prefix_len * hd;
  const size_t es = esize(m->et);
  if (m->tern) {
    QuantArgs q{};
    q.M = M; q.K = K; q.x = prefix_hidden; q.ldx = K; q.src_type = 1; q.q = w->q8; q.r = w->r8;
    HIP_TRY(launch_quantize(q, s));
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
        const Tiling t = gemm_tiling(m->et, M, N, K, 1);
        g.ks = t.nc * gemm_chunk_k(m->et); g.nsplit = t.nsplit; g.n_tiles = t.n_tiles;
        g.ws = w->ws; g.cnt = w->cnt;
        HIP_TRY(launch_gemm(m->et, t.ms, 1, t.nc, g, t.units, s));
      } else {
        TernArgs ta{};
        const Tiling t = tern_tiling(M, N, K, 1);
        ta.M = M; ta.N = N; ta.K = K; ta.x = w->q8; ta.w = (const uint8_t*)sw.kvc; ta.rscale = w->r8;
        ta.wscale = sw.s_kvc; ta.ks = t.nc * 256; ta.nsplit = t.nsplit; ta.n_tiles = t.n_tiles;
        ta.ws = reinterpret_cast<int*>(w->ws); ta.cnt = w->cnt; ta.e = g;
        HIP_TRY(launch_ternary_gemm(ta, t.ms, t.units, s));
      }
    }
  return VLA_OK;
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
  if ((long long)batch * c.n_action > 65536) return fail(VLA_E_UNSUPPORTED, "batch * n_action too large");
  if (n_steps < 1 || n_steps > VLA_MAX_STEPS) return fail(VLA_E_SHAPE, "n_steps %d not in 1..%d", n_steps, VLA_MAX_STEPS);
  if (c.head_regression && n_steps != 1) return fail(VLA_E_SHAPE, "the regression head takes n_steps == 1");
  if (kv_cache_bytes != vla_kv_cache_bytes(m, batch, prefix_len))
    return fail(VLA_E_SHAPE, "kv_cache_bytes %zu != %zu for batch %d, prefix_len %d", kv_cache_bytes,
                vla_kv_cache_bytes(m, batch, prefix_len), batch, prefix_len);
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

  auto key = std::make_tuple(batch, prefix_len, n_steps);
  auto it = m->plans.find(key);
  Plan* p;
  if (it == m->plans.end()) {
    if (m->plans.size() >= 8) m->plans.erase(m->plans.begin());
    std::unique_ptr<Plan> np(new Plan());
    np->B = batch;
    np->P = prefix_len;
    np->T = n_steps;
    VLA_TRY(build_plan(m, np.get()));
    p = np.get();
    m->plans[key] = std::move(np);
  } else {
    p = it->second.get();
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(launch_set_params(p->cp, cpv, s));
  if (m->loop_mode == 0) {
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
  a.ks = t.nc * 256; a.nsplit = t.nsplit; a.n_tiles = t.n_tiles;
  if (a.nsplit > 1) HIP_TRY(launch_fill_u32(reinterpret_cast<unsigned*>(acc_out), 0u, (size_t)M * N, s));
  HIP_TRY(launch_ternary_gemm(a, t.ms, t.units, s));
  return VLA_OK;
}

// ---- test entries ----------------------------------------------------------

vla_status vla_test_gemm(int32_t elem, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                         int32_t force_nsplit, float* y, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  if (!x || !w || !y || !al16(x) || !al16(w) || !al16(y)) return fail(VLA_E_ARG, "bad buffer");
  if (M < 1 || N < 1 || K < 1 || K % (elem ? 8 : 4)) return fail(VLA_E_SHAPE, "bad GEMM shape");
  const int et = elem ? ET_BF16 : ET_F32;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Tiling t = gemm_tiling(et, M, N, K, 1, force_nsplit);
  GemmArgs g{};
  g.M = M; g.N = N; g.K = K; g.X = x; g.ldx = K; g.W = w;
  g.ks = t.nc * gemm_chunk_k(et); g.nsplit = t.nsplit; g.n_tiles = t.n_tiles;
  g.epi = EPI_STORE; g.out = y; g.ldo = N; g.out_f32 = 1;
  float* ws = nullptr;
  unsigned* cnt = nullptr;
  if (t.nsplit > 1) {
    HIP_TRY(hipMalloc(&ws, (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, 1) * 4));
    HIP_TRY(hipMalloc(&cnt, (size_t)t.m_tiles * t.n_tiles * 4));
    HIP_TRY(hipMemset(cnt, 0, (size_t)t.m_tiles * t.n_tiles * 4));
  }
  g.ws = ws; g.cnt = cnt;
  hipError_t e = launch_gemm(et, t.ms, 1, t.nc, g, t.units, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(ws);
  (void)hipFree(cnt);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "gemm: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

vla_status vla_test_attention(int32_t elem, int32_t mode, const void* q, const void* k_self, const void* v_self,
                              const void* k_cache, const void* v_cache, int32_t B, int32_t n, int32_t P, int32_t H,
                              int32_t G, int32_t hd, int32_t kv_split, void* o, void* stream) {
  if (elem != 0 && elem != 1) return fail(VLA_E_ARG, "elem must be 0 or 1");
  if (mode < 0 || mode > 2) return fail(VLA_E_ARG, "mode must be 0, 1 or 2");
  if (!q || !o || (mode != 1 && (!k_self || !v_self)) || (mode != 0 && (!k_cache || !v_cache)))
    return fail(VLA_E_ARG, "NULL buffer");
  if (B < 1 || n < 1 || (mode != 0 && P < 1) || H < 1 || G < 1 || H % G) return fail(VLA_E_SHAPE, "bad shape");
  if (!(hd == 64 || hd == 128 || (elem == 1 && hd == 256))) return fail(VLA_E_UNSUPPORTED, "head_dim");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  AttnArgs a{};
  a.mode = mode; a.B = B; a.n = n; a.P = mode == 0 ? 0 : P; a.H = H; a.G = G; a.hd = hd;
  a.q = q; a.ldq = H * hd; a.ks = k_self; a.vs = v_self; a.ldkv = G * hd;
  a.kc = k_cache; a.vc = v_cache; a.o = o; a.ldo = H * hd; a.scale = 1.0f / std::sqrt((float)hd);
  const int total = (mode == 0 ? 0 : P) + (mode == 1 ? 0 : n);
  const int QT = cdiv(n, 16);
  int split = kv_split > 0 ? kv_split : std::max(1, std::min(cdiv(256, B * H * QT), cdiv(total, 32)));
  a.key_chunk = cdiv(cdiv(total, split), 32) * 32;
  a.kv_split = cdiv(total, a.key_chunk);
  float* ws = nullptr;
  unsigned* cnt = nullptr;
  if (a.kv_split > 1) {
    HIP_TRY(hipMalloc(&ws, attention_ws_floats(a) * 4));
    HIP_TRY(hipMalloc(&cnt, (size_t)B * H * QT * 4));
    HIP_TRY(hipMemset(cnt, 0, (size_t)B * H * QT * 4));
  }
  a.ws = ws; a.cnt = cnt;
  hipError_t e = launch_attention(elem ? ET_BF16 : ET_F32, a, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(ws);
  (void)hipFree(cnt);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "attention: %s", hipGetErrorString(e != hipSuccess ? e : e2));
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

vla_status vla_test_ternary_linear(const float* x, const uint8_t* w_packed, int32_t M, int32_t N, int32_t K,
                                   float scale, float* y, void* stream) {
  if (!x || !w_packed || !y || !al16(x) || !al16(w_packed) || !al16(y)) return fail(VLA_E_ARG, "bad buffer");
  if (M < 1 || N < 1 || K < 64 || K % 64 || K > 16384) return fail(VLA_E_SHAPE, "bad shape");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Tiling t = tern_tiling(M, N, K, 1);
  int8_t* q8 = nullptr;
  float *r8 = nullptr, *sc = nullptr, *ws = nullptr;
  unsigned* cnt = nullptr;
  HIP_TRY(hipMalloc(&q8, (size_t)M * K));
  HIP_TRY(hipMalloc(&r8, (size_t)M * 4));
  HIP_TRY(hipMalloc(&sc, (size_t)N * 4));
  std::vector<float> hs(N, scale);
  HIP_TRY(hipMemcpy(sc, hs.data(), (size_t)N * 4, hipMemcpyHostToDevice));
  if (t.nsplit > 1) {
    HIP_TRY(hipMalloc(&ws, (size_t)t.m_tiles * t.n_tiles * t.nsplit * gemm_ws_floats_per_unit(t.ms, 1) * 4));
    HIP_TRY(hipMalloc(&cnt, (size_t)t.m_tiles * t.n_tiles * 4));
    HIP_TRY(hipMemset(cnt, 0, (size_t)t.m_tiles * t.n_tiles * 4));
  }
  QuantArgs qa{};
  qa.M = M; qa.K = K; qa.x = x; qa.ldx = K; qa.src_type = 0; qa.q = q8; qa.r = r8;
  TernArgs a{};
  a.M = M; a.N = N; a.K = K; a.x = q8; a.w = w_packed; a.rscale = r8; a.wscale = sc;
  a.ks = t.nc * 256; a.nsplit = t.nsplit; a.n_tiles = t.n_tiles;
  a.ws = reinterpret_cast<int*>(ws); a.cnt = cnt;
  a.e.M = M; a.e.N = N; a.e.K = K; a.e.epi = EPI_STORE; a.e.out = y; a.e.ldo = N; a.e.out_f32 = 1;
  hipError_t e = launch_quantize(qa, s);
  if (e == hipSuccess) e = launch_ternary_gemm(a, t.ms, t.units, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(q8); (void)hipFree(r8); (void)hipFree(sc); (void)hipFree(ws); (void)hipFree(cnt);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(VLA_E_DEVICE, "ternary linear: %s", hipGetErrorString(e != hipSuccess ? e : e2));
  return VLA_OK;
}

}  // extern "C"

// Internal interfaces between the host runtime (vla_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#define VLA_MAX_STEPS 64

enum ElemType { ET_F32 = 0, ET_BF16 = 1 };
enum Act { ACT_NONE = 0, ACT_SILU = 1, ACT_GELU = 2, ACT_RELU2 = 3 };

// Per-call values of vla_denoise, written to device memory by a tiny kernel
// before the (possibly graph-replayed) launch sequence so that the sequence
// itself never changes between calls.
struct CallParams {
  const void* kv_cache;
  const float* noise;
  const float* state;
  float* actions_out;
  const float* act_mean;
  const float* act_std;
  float tau[VLA_MAX_STEPS + 1];
};

// GEMM epilogues, applied to y = X W^T after the split-K reduction.
enum GemmEpi {
  EPI_STORE = 0,    // out[m][n] = act(y + bias[n]) in the element type or fp32
  EPI_RESID = 1,    // x[m][n] += alpha[n] * y
  EPI_GLU = 2,      // W rows interleaved gate/up in blocks of 16: h = act(g) * u
  EPI_EULER = 3,    // v = y + bias; a += dt v (or a = v); last step: denormalised output
  EPI_KVCACHE = 4,  // scatter [rows of one request][K|V][G][hd] into the cache layout
  EPI_PARTIAL = 5,  // raw fp32 split-K partial: out[split][m][n]
};

struct GemmArgs {
  // problem
  int M, N, K;
  const void* X;
  int ldx;
  const void* W;           // [N][K] row-major in the element type
  int n_tiles;             // tiles along N (set by the launcher)
  int m_tiles;             // tiles along M (tiled kernel; set by the launcher)
  int nsplit;              // K-splits (set by the launcher; > 1 only with EPI_PARTIAL)
  int kper;                // K-range of one split (skinny kernel; set by the launcher)
  // epilogue
  int epi;
  int act;
  const float* bias;
  void* out;               // EPI_STORE / EPI_GLU destination
  int ldo;
  int out_f32;             // EPI_STORE: 1 = fp32 output, 0 = element type
  float* xres;             // EPI_RESID residual [M][ldxr]
  int ldxr;
  const float* alpha;
  // EPI_EULER
  float* a;                // [M][N]
  const CallParams* cp;
  int step;
  int regression;
  int last;
  int stok;                // tokens per request when row 0 of each request is a state token (no
                           // action output: skipped; action row = b (stok-1) + t-1), else 0
  // EPI_KVCACHE: row m = b*P + p, column n = slot*lay_cols + kv*d_kv + g*hd + c
  void* cache;             // base of cache slot 0: [slots][2][B][G][P][hd]
  int P, hd, d_kv, B;
  int lay_cols;            // columns per cache slot (2 d_kv) when one GEMM fills several slots, else 0
  size_t lay_stride;       // elements per cache slot
};

struct AttnArgs {
  int mode;                // 0 self, 1 cross, 2 joint
  int B, n, P;             // requests, action tokens, prefix rows
  int H, G, hd;
  const void* q;           // [B*n][ldq], head h at column h*hd
  int ldq;
  const void* ks;          // self keys   [B*n][ldkv], head g at column g*hd
  const void* vs;          // self values
  int ldkv;
  const void* kc;          // cache K of this layer: [B][G][P][hd]; NULL -> from cp
  const void* vc;
  const CallParams* cp;    // kv_cache base when kc == NULL
  size_t layer_off;        // element offset of this layer's K block in the cache
  void* o;                 // [B*n][ldo]
  int ldo;
  float scale;
  int kv_split;            // key splits
  int hsplit;              // groups of query heads per K/V head (workgroups per group)
  int key_chunk;           // 32-key blocks per split (64-key blocks when tiled)
  int tiled;               // 1: the 128-row tiled kernel (bf16, large query counts)
  int causal;              // self / joint: query t sees action keys 0 .. t only (prefix rows all)
  void* part;              // [kv_split][B*n][H*hd] per-split output (kv_split > 1)
  float* stats;            // [kv_split][B*n][H][2] per-split (max, sum)
};

struct QuantArgs {
  int M, K;
  const void* x;           // [M][ldx] fp32 or bf16
  int ldx;
  int src_type;            // 0 fp32, 1 bf16
  int8_t* q;               // [M][K]
  float* r;                // [M]
};

// Per-row residual finish + adaRMS of the next sublayer:
//   x[m] = x[m] + alpha * sum_s part[s][m]      (mode 0; nsplit may be 0)
//   x[m] = a[m] W_in^T + xs[b] + E_pos[token]    (mode 1, the input embedding)
//   u[m] = x[m] / sqrt(mean(x[m]^2) + eps) * (1 + gamma) + beta
struct RowNormArgs {
  int mode;                // 0: residual stream x (+ alpha * sum of partials); 1: input embedding;
                           // 2: x = x_in (element type), the first norm of a backbone prefill
  int M, d;
  float* x;                // [M][d]
  const float* part;       // [nsplit][M][d]
  int nsplit;
  const float* alpha;      // [d] or NULL (no residual update)
  const float* a;          // mode 1: [M][A]
  const void* W_in;        // [d][A]
  const float* xs;         // [B][d]
  const void* E_pos;       // [n][d]
  int n, A;                // n: token rows per request
  int stok;                // mode 1, state-token variant: row 0 of a request = xs, action row t
                           // (t >= 1) = b_in + E_pos[t-1] + a W_in; 0 = xs + E_pos + a W_in
  const float* b_in;
  const float* gamma;
  const float* beta;
  float eps;
  void* u;                 // [M][d] element type (u_f32 = 0) or fp32
  int u_f32;
  int8_t* q;               // if set (u_f32 = 1): also the int8 absmax quantisation of u, [M][d]
  float* qr;               // and its per-row absmax [M]
  const void* x_in;        // mode 2: [M][d] element type
};

struct TernArgs {
  int M, N, K;
  const int8_t* x;         // [M][K]
  const uint8_t* w;        // [N][K/4] packed
  const float* rscale;     // [M] absmax per row (dequant) or NULL for raw acc
  const float* wscale;     // [N] per W-row scale (the per-tensor scale of its matrix)
  int32_t* acc_out;        // raw int32 output (when rscale == NULL); zero-filled if nsplit > 1
  int ks, nsplit, n_tiles;  // nsplit > 1 only for the raw int32 output (atomic accumulation)
  int m_tiles;              // tiled kernel: row tiles (set by its launcher)
  // dequantised epilogue (same meaning as GemmArgs)
  GemmArgs e;
};

// Launch shapes of the two dense GEMM kernels (chosen on the host).
struct SkinnyShape {
  int ms, nsub, cpw, nsplit, kper, n_tiles, m_tiles, units;
  size_t lds;
};
struct WideShape {
  int ms, nsub, nc, n_tiles, m_tiles, units;
  size_t lds;
};
// Tiled kernel: a (32*ms) x (32*ns) output tile per workgroup, K split in
// nsplit ranges of kper.  grid = units rounded up to a multiple of 8.
struct TileShape {
  int ms, ns, nsplit, kper, n_tiles, m_tiles, units, grid;
  size_t lds;
};

// Persistent tensor-parallel denoise loop (bf16, joint attention, batch 1):
// weights of one layer, library-owned.
struct PLayer {
  const void* wqkv;          // [d_q + 2 d_kv][d]
  const void* wo;            // [d][d_q]
  const void* wgu;           // GLU: gate/up interleaved in 16-row blocks [2F][d]; GELU: W1 [F][d]
  const void* wd;            // [8][d][F / 8]: team t's columns of W_d [d][F] as one block
  size_t cache_off;          // element offset of this layer's K block in the cache
};

struct PersistArgs {
  int L, d, H, G, hd, F, n, P, A, T;
  int glu, act;              // MLP form: gate/up pair (1) or single W1 (0); activation
  int HT;                    // query heads per team (H / 8)
  int kba, nsplit;           // attention: 32-key blocks per split, key splits
  float eps, scale;
  const PLayer* layers;      // [L] (device)
  const CallParams* cp;
  const float* mods;         // [T][L * 2 * 3 * d]: per sublayer gamma, beta, alpha
  const float* modf;         // [T][2 d]: final gamma, beta
  const void* w_in;          // [d][A]
  const float* xs;           // [d]: b_in + b_s + state W_s^T
  const void* e_pos;         // [n][d]
  const void* w_out;         // [A][d]
  const float* b_out;        // [A]
  const float* a0;           // [n][A]: the noise chunk a_0
  // team-replicated workspace (team = one of 8 groups of 32 workgroups)
  void* u;                   // [8][n][d]
  void* qkv;                 // [8][n][(HT + 2) hd]: team heads' Q, the team's K, V
  void* apart;               // [8][nsplit][n][HT hd]
  float* astat;              // [8][nsplit][n][HT][2]
  void* omerged;             // [8][n][HT hd]: merged attention output of the team's heads
  void* hbuf;                // [8][n][F / 8]
  float* delta;              // [2][8][n][d]: per-team partial residual updates
  unsigned* sync;            // PERSIST_SYNC_WORDS words (barrier flags, rank counters, error word), zero at launch
  int* err;                  // = sync + PERSIST_ERR_OFF: set when a barrier times out
  long spin_limit;           // polls of one barrier wait before it gives up (sets *err)
  // optional phase timeline: workgroup 0 of each team records the 100 MHz
  // clock before and after every barrier, PERSIST_TRACE_MAX entries per team
  unsigned long long* trace;
  int trace_all;             // 1: every workgroup records its first PERSIST_TRACE_WG marks (row team * 32 + rank)
};
// Grid barrier flags [8][32] in 8 copies, 4 KB apart (team x polls copy x);
// the first copy's 4 KB also holds the rank counters, the error word and the
// team barrier flags.
constexpr int PERSIST_GFLAG_STRIDE = 1024;        // words between two copies of the grid flags
constexpr int PERSIST_RANK_OFF = 8 * 32;          // 8 per-XCD arrival counters (team ranks)
constexpr int PERSIST_ERR_OFF = 8 * 32 + 32;      // the error word, on a line of its own
constexpr int PERSIST_TFLAG_OFF = 8 * 32 + 64;    // team barrier flags [8][32], one 128-byte line per team
constexpr int PERSIST_SYNC_WORDS = 8 * PERSIST_GFLAG_STRIDE;
constexpr long PERSIST_SPIN_DEFAULT = 1L << 20;   // barrier polls before a timeout (about 0.25 s)
constexpr int PERSIST_TRACE_MAX = 8192;
constexpr int PERSIST_TRACE_WG = 8 * PERSIST_TRACE_MAX / 256;   // marks per workgroup when all record
constexpr int PERSIST_MAX_LAYERS = 64;

// ---- launchers (each enqueues on `s`, returns hipError_t) ----
int gemm_chunk_k(int et);  // K covered by one chunk (all 4 lane groups of a wave)
bool skinny_plan(int et, int M, int N, int K, int nsub, bool allow_split, SkinnyShape* sh);
void wide_plan(int et, int M, int N, int K, int nsub, WideShape* sh);
hipError_t launch_gemm_skinny(int et, const SkinnyShape& sh, GemmArgs a, hipStream_t s);
hipError_t launch_gemm_wide(int et, const WideShape& sh, GemmArgs a, hipStream_t s);
// Tiled bf16 kernel for M > 128.  force < 0: the cost model picks the tile and
// the K-split (split only if allow_split); force = 0..3 fixes the tile
// (64x128, 128x128, 256x128, 128x256) with no split.  False if not applicable.
bool tile_plan(int et, int M, int N, int K, bool allow_split, int force, TileShape* sh);
hipError_t launch_gemm_tile(const TileShape& sh, GemmArgs a, hipStream_t s);

// which: 0 = key-split kernel and (when kv_split > 1) the merge, 1 = the
// key-split kernel only, 2 = the merge only.
hipError_t launch_attention(int et, const AttnArgs& a, hipStream_t s, int which = 0);
// want_splits / want_hsplit 0 = automatic (at most 4 heads per workgroup,
// about 224 workgroups)
void attention_split(AttnArgs& a, int want_splits, int want_hsplit = 0);
// The 128-row tiled attention kernel: whether the runtime picks it for this
// shape, and its split plan (want_splits 0 = about one workgroup per CU).
bool attention_tile_eligible(int et, const AttnArgs& a);
void attention_tile_split(AttnArgs& a, int want_splits);
int attention_max_blocks();  // most 32-key blocks (prefix blocks + action blocks) one call handles
size_t attention_part_bytes(int et, const AttnArgs& a);
size_t attention_stats_bytes(const AttnArgs& a);

hipError_t launch_set_params(CallParams* dst, const CallParams& src, hipStream_t s);
// Chunk start: a <- noise and xs (per-request constant embedding) for B
// requests, plus the time embedding rows e[Tpad][d] when e is not null.
hipError_t launch_chunk_start(int et, const CallParams* cp, float* a, float* xs, const void* W_s,
                              const float* b_s, const float* b_in, int B, int n, int A, int S, int d, void* e,
                              int T, int Tpad, hipStream_t s);
hipError_t launch_row_norm(int et, const RowNormArgs& a, hipStream_t s);
hipError_t launch_time_embed(int et, const CallParams* cp, void* e, int T, int Tpad, int d, hipStream_t s);
hipError_t launch_copy_f32(float* dst, const float* src, size_t n, hipStream_t s);
hipError_t launch_quantize(const QuantArgs& a, hipStream_t s);
hipError_t launch_ternary_dot4(const TernArgs& a, hipStream_t s);   // VALU sdot4 variant (EPI_STORE)
// The tiled W2A8 kernel takes the shape (many token rows, K % 128 == 0).
bool tern_tile_eligible(int M, int N, int K);
// The tiled W2A8 kernel with (32 ms)-row tiles (ms 1, 2 or 4) on `waves`
// waves: kgroups 1 = waves of 32 columns each (4, or 8 with ms 2 or 4 for a
// 256-column tile); kgroups 2 = eight waves of a 128-column tile in two
// groups taking alternate K-slices.  The same sums as every other
// configuration; hipErrorInvalidValue for shapes or tiles it does not take.
hipError_t launch_ternary_tile(const TernArgs& a, int ms, int waves, int kgroups, hipStream_t s);
hipError_t launch_ternary_gemm(const TernArgs& a, int ms, int units, hipStream_t s);
hipError_t launch_check_finite(const float* x, size_t n, int* flag, hipStream_t s);
hipError_t launch_fill_u32(unsigned* p, unsigned v, size_t n, hipStream_t s);
hipError_t launch_sum_partials(float* y, const float* part, int nsplit, size_t n, hipStream_t s);
// rotary position embedding in place (rotate-half); positions pos0 + row % rpr
hipError_t launch_rope(int et, void* x, int rows, int rpr, int ld, int col0, int nheads, int hd, int pos0, float base,
                       hipStream_t s);
// Persistent kernel: whether a shape is supported, the dynamic LDS it needs,
// and the cooperative launch (256 workgroups of 512 threads).
bool persist_supported(int d, int hd, int H, int G, int F, int n, int P, int A, int glu, int* kba, int* nsplit);
// The device can hold every workgroup of the persistent kernel at once (its
// 256 workgroups, one per compute unit, 32 on each of the 8 XCDs).
bool persist_resident(int d, int hd, int HT);
size_t persist_lds_bytes(int hd, int HT);
hipError_t launch_persist(const PersistArgs& a, hipStream_t s);

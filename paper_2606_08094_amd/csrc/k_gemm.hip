// MFMA GEMMs y = X W^T for the expert's projections.  No workgroup ever
// waits on another: an output tile is reduced inside one workgroup, or written
// as a split-K partial that a later launch adds up (on this 8-XCD part an
// agent-scope fence writes back and invalidates the XCD's whole L2, so
// in-kernel cross-workgroup reductions cost far more than a launch).
//
// gemm_skinny -- the per-step projections, M <= 128 token rows.
//   A workgroup of 8 waves owns 16*NSUB rows of W (NSUB = 2: a gate/up pair
//   of interleaved 16-row blocks), up to 16*MS token rows and one K-range
//   (split-K across workgroups when the grid would otherwise not fill the
//   chip).  The K-range is cut into chunks of KC k-values; wave w takes
//   chunks w, w+8, ... (CPW per round).  Every operand goes straight from
//   global memory into MFMA-layout registers: a round issues all W and X
//   loads of the wave before the first MFMA, so a workgroup pays one memory
//   latency per round instead of one per staging step.  The eight partial
//   tiles are summed in wave order through LDS and waves 0..MS-1 run the
//   epilogue of one 16-row subtile each.
//
// gemm_wide -- fp32 with M > 128.  Four waves along N (NT = 64*NSUB), X
//   staged per K-slice in LDS and shared by the four waves, K-slices looped
//   inside the workgroup.
//
// gemm_tile -- bf16 with M > 128 (batched requests, the prefix K/V build),
//   where the work is MFMA-bound.  Four waves (2 x 2) own a BM x BN output tile
//   (BM = 32*MS, BN = 32*NS); X and W are both staged through LDS in K-slices
//   of 64, double-buffered: the global loads of slice s+1 are in flight while
//   the MFMAs of slice s run, and one barrier per slice separates the two
//   buffers.  LDS rows are padded by 16 bytes so that the rows of one MFMA
//   operand load fall in distinct banks.  Tiles along M are numbered fastest
//   and blocks are renumbered so that consecutive tiles (which share one W
//   slice) run on the same XCD and its L2.
//
// Operand layout: in a chunk, lane l of a wave reads 16-byte vector v of row
// (l % 16) at k-offset v*4*E + (l/16)*E, for W and X alike, so the MFMA's k
// order is a permutation common to both operands and every load instruction
// of a wave reads 64 contiguous bytes per row.
#include <algorithm>
#include <cmath>
#include <utility>

#include "gemm_epilogue.h"

namespace {

constexpr int VPL = 4;   // 16-byte vectors per lane per chunk
constexpr int WKS = 8;   // waves of a skinny workgroup

// Stage X rows m0 .. m0+MT-1, columns k0 .. k0+KW-1 (KW a multiple of E) into
// LDS with row pitch `pitch` elements; zeros outside [M] x [K].  A thread
// issues the loads of up to UB items before storing any of them.
template <typename T, int MT>
VLA_DEV void stage_x(const GemmArgs& a, T* xs, int pitch, int m0, int k0, int KW) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int UB = 8;
  const int vrow = KW / E;
  const int total = MT * vrow;
  const int nthr = blockDim.x;
  const T* X = reinterpret_cast<const T*>(a.X);
  for (int base = threadIdx.x; base < total; base += UB * nthr) {
    uint4 v[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int i = base + u * nthr;
      const int row = i / vrow, kv = i - row * vrow;
      const bool ok = i < total && (m0 + row) < a.M && (k0 + kv * E) < a.K;
      v[u] = ok ? ldg16(X + (size_t)(m0 + row) * a.ldx + k0 + kv * E) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int i = base + u * nthr;
      if (i < total) {
        const int row = i / vrow, kv = i - row * vrow;
        *reinterpret_cast<uint4*>(xs + (size_t)row * pitch + kv * E) = v[u];
      }
    }
  }
}

// ---------------------------------------------------------------------------
template <typename T, int MS, int NSUB, int CPW>
__global__ __launch_bounds__(64 * WKS) void gemm_skinny(GemmArgs a) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int KC = 4 * VPL * E;
  extern __shared__ __align__(16) unsigned char smem[];
  f32x4* red = reinterpret_cast<f32x4*>(smem);  // [WKS][MS][NSUB][64]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  int bid = blockIdx.x;
  const int split = bid % a.nsplit;
  bid /= a.nsplit;
  const int ntile = bid % a.n_tiles, mtile = bid / a.n_tiles;
  const int m0 = mtile * 16 * MS;
  const int nb = ntile * 16 * NSUB;
  const int k0 = split * a.kper;
  const int k1 = min(K, k0 + a.kper);
  const int nck = (k1 - k0 + KC - 1) / KC;
  const T* W = reinterpret_cast<const T*>(a.W);
  const T* X = reinterpret_cast<const T*>(a.X);

  f32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c0 = 0; c0 < nck; c0 += WKS * CPW) {
    uint4 wreg[CPW][NSUB][VPL];
    uint4 xreg[CPW][MS][VPL];
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int c = c0 + wave + j * WKS;
      const int kc = k0 + c * KC + g4 * E;
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        const int n = nb + s * 16 + r16;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const int k = kc + v * 4 * E;
          wreg[j][s][v] = (c < nck && n < N && k < k1) ? ldg16(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int c = c0 + wave + j * WKS;
      const int kc = k0 + c * KC + g4 * E;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int m = m0 + ms * 16 + r16;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const int k = kc + v * 4 * E;
          xreg[j][ms][v] = (c < nck && m < M && k < k1) ? ldg16(X + (size_t)m * a.ldx + k) : make_uint4(0, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j)
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
          for (int v = 0; v < VPL; ++v) mma16(acc[ms][s], xreg[j][ms][v], wreg[j][s][v], T());
  }

  // sum the eight partial tiles in wave order; wave ms < MS finishes subtile ms
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) red[((wave * MS + ms) * NSUB + s) * 64 + lane] = acc[ms][s];
  __syncthreads();
  if (wave >= MS) return;
  f32x4 r[1][NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    r[0][s] = red[((0 * MS + wave) * NSUB + s) * 64 + lane];
#pragma unroll
    for (int w = 1; w < WKS; ++w) r[0][s] += red[((w * MS + wave) * NSUB + s) * 64 + lane];
  }
  wave_epilogue<T, 1, NSUB>(a, r, m0 + wave * 16, nb, split);
}

// ---------------------------------------------------------------------------
template <typename T, int MS, int NSUB, int NC>
__global__ __launch_bounds__(256) void gemm_wide(GemmArgs a) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int KCL = VPL * E;
  constexpr int KC = 4 * KCL;
  constexpr int KS = NC * KC;
  constexpr int MT = 16 * MS;
  constexpr int NT = 64 * NSUB;
  constexpr int PITCH = KS + E;
  extern __shared__ __align__(16) unsigned char smem[];
  T* xs = reinterpret_cast<T*>(smem);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int N = a.N, K = a.K;
  const int ntile = blockIdx.x % a.n_tiles, mtile = blockIdx.x / a.n_tiles;
  const int m0 = mtile * MT;
  const int nb = ntile * NT + wave * 16 * NSUB;
  const T* W = reinterpret_cast<const T*>(a.W);

  f32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K; k0 += KS) {
    uint4 wreg[NSUB][NC][VPL];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int n = nb + s * 16 + r16;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const int k = k0 + c * KC + g4 * KCL + v * E;
          wreg[s][c][v] = (n < N && k < K) ? ldg16(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
        }
    }
    if (k0 > 0) __syncthreads();  // previous slice's LDS reads done
    stage_x<T, MT>(a, xs, PITCH, m0, k0, KS);
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (k0 + c * KC >= K) break;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const T* xrow = xs + (size_t)(ms * 16 + r16) * PITCH + c * KC + g4 * KCL;
        uint4 xf[VPL];
#pragma unroll
        for (int v = 0; v < VPL; ++v) xf[v] = *reinterpret_cast<const uint4*>(xrow + v * E);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
          for (int v = 0; v < VPL; ++v) mma16(acc[ms][s], xf[v], wreg[s][c][v], T());
      }
    }
  }
  wave_epilogue<T, MS, NSUB>(a, acc, m0, nb, 0);
}


// ---------------------------------------------------------------------------
constexpr int TBK = 64;           // K-slice of gemm_tile
constexpr int TPITCH = TBK + 8;   // LDS row pitch in elements (16 bytes of padding)

// LDS of gemm_tile_rs: two K-slice buffers of X and W rows, reused for the
// fp32 output tile by the epilogue.
template <int MS, int NS>
constexpr size_t tile_lds_bytes() {
  const size_t stage = (size_t)2 * (32 * MS + 32 * NS) * TPITCH * sizeof(bf16_t);
  const size_t out = (size_t)(32 * MS) * (32 * NS + 4) * sizeof(float);
  return stage > out ? stage : out;
}


// Epilogue of the tiled kernels over the fp32 tile ct [BM][CP] (rows m0..,
// columns n0..): each thread finishes 4 consecutive columns of a row, so a row
// is written with 8- or 16-byte stores.  For EPI_GLU the tile's columns are
// 16-row blocks of gate and up rows in turn, and output column f pairs gate
// column (f/16)*32 + f%16 with the up column 16 further on.
VLA_DEV void store4(float* p, float4 v, bool vec) {
  if (vec) *reinterpret_cast<float4*>(p) = v;
  else { p[0] = v.x; p[1] = v.y; p[2] = v.z; p[3] = v.w; }
}
VLA_DEV void store4(bf16_t* p, float4 v, bool vec) {
  if (vec) *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
  else { p[0] = f2bf(v.x); p[1] = f2bf(v.y); p[2] = f2bf(v.z); p[3] = f2bf(v.w); }
}
// Columns c .. c+3 of which only the first `n` exist.
template <typename T>
VLA_DEV void store4n(T* p, float4 v, int n, bool vec) {
  if (n >= 4) { store4(p, v, vec); return; }
  const float e[4] = {v.x, v.y, v.z, v.w};
  for (int j = 0; j < n; ++j) {
    if constexpr (sizeof(T) == 4) p[j] = e[j]; else p[j] = f2bf(e[j]);
  }
}
VLA_DEV float4 act4(int act, float4 v) { return make_float4(act_f(act, v.x), act_f(act, v.y), act_f(act, v.z), act_f(act, v.w)); }

// Runs f(m, n, nv, v) for every 4-column group of the tile's first `rows`
// rows (nv = columns left in the matrix from n, v = the tile's 4 values; for
// GLU the 4 gate and 4 up values come as g and u).  The loop is unrolled with
// every LDS read issued before the first store.
template <int RP, int BN, int CP, int NT, typename Fn>
VLA_DEV void epi_rows(const float* ct, int rows, int n0, int N, Fn&& f) {
  constexpr int TPR = BN / 4, IT = (RP * TPR + NT - 1) / NT;
  float4 v[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx / TPR, c = (idx % TPR) * 4;
    v[j] = (r < RP) ? *reinterpret_cast<const float4*>(ct + r * CP + c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx / TPR, c = (idx % TPR) * 4;
    if (r < rows && n0 + c < N) f(r, n0 + c, N - (n0 + c), v[j]);
  }
}
template <int RP, int BN, int CP, int NT, typename Fn>
VLA_DEV void epi_rows_glu(const float* ct, int rows, int f0, int F, Fn&& f) {
  constexpr int TPR = BN / 8, IT = (RP * TPR + NT - 1) / NT;
  float4 g[IT], u[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx / TPR, c = (idx % TPR) * 4;
    const int cg = (c >> 4) * 32 + (c & 15);
    g[j] = (r < RP) ? *reinterpret_cast<const float4*>(ct + r * CP + cg) : make_float4(0.f, 0.f, 0.f, 0.f);
    u[j] = (r < RP) ? *reinterpret_cast<const float4*>(ct + r * CP + cg + 16) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx / TPR, c = (idx % TPR) * 4;
    if (r < rows && f0 + c < F) f(r, f0 + c, F - (f0 + c), g[j], u[j]);
  }
}

template <int RP, int BN, int CP, int NT = 256>
VLA_DEV void tile_epilogue(const GemmArgs& a, const float* ct, int m0, int n0, int split) {
  const int M = a.M, N = a.N;
  const int rows = min(RP, M - m0);
  if (rows <= 0) return;
  switch (a.epi) {
    case EPI_GLU: {
      const bool vec = (a.ldo & 3) == 0;
      const int act = a.act;
      auto f = [&](int r, int fc, int nv, float4 g, float4 u) {
        const float4 gg = act4(act, g);
        const float4 h = make_float4(gg.x * u.x, gg.y * u.y, gg.z * u.z, gg.w * u.w);
        const size_t o = (size_t)(m0 + r) * a.ldo + fc;
        if (a.out_f32) store4n(reinterpret_cast<float*>(a.out) + o, h, nv, vec);
        else store4n(reinterpret_cast<bf16_t*>(a.out) + o, h, nv, vec);
      };
      epi_rows_glu<RP, BN, CP, NT>(ct, rows, n0 / 2, N / 2, f);
      break;
    }
    case EPI_STORE: {
      const bool vec = (a.ldo & 3) == 0;
      auto f = [&](int r, int n, int nv, float4 v) {
        if (a.bias) {
          const float b[4] = {a.bias[n], nv > 1 ? a.bias[n + 1] : 0.f, nv > 2 ? a.bias[n + 2] : 0.f,
                              nv > 3 ? a.bias[n + 3] : 0.f};
          v = make_float4(v.x + b[0], v.y + b[1], v.z + b[2], v.w + b[3]);
        }
        v = act4(a.act, v);
        const size_t o = (size_t)(m0 + r) * a.ldo + n;
        if (a.out_f32) store4n(reinterpret_cast<float*>(a.out) + o, v, nv, vec);
        else store4n(reinterpret_cast<bf16_t*>(a.out) + o, v, nv, vec);
      };
      epi_rows<RP, BN, CP, NT>(ct, rows, n0, N, f);
      break;
    }
    case EPI_PARTIAL: {
      float* out = reinterpret_cast<float*>(a.out) + (size_t)split * M * a.ldo;
      const bool vec = (a.ldo & 3) == 0;
      auto f = [&](int r, int n, int nv, float4 v) { store4n(out + (size_t)(m0 + r) * a.ldo + n, v, nv, vec); };
      epi_rows<RP, BN, CP, NT>(ct, rows, n0, N, f);
      break;
    }
    case EPI_RESID: {
      auto f = [&](int r, int n, int nv, float4 v) {
        float* xp = a.xres + (size_t)(m0 + r) * a.ldxr + n;
        const float e[4] = {v.x, v.y, v.z, v.w};
        for (int j = 0; j < 4 && j < nv; ++j) xp[j] = xp[j] + a.alpha[n + j] * e[j];
      };
      epi_rows<RP, BN, CP, NT>(ct, rows, n0, N, f);
      break;
    }
    case EPI_KVCACHE: {
      const int G = a.d_kv / a.hd;
      auto f = [&](int r, int n, int nv, float4 v) {
        const int m = m0 + r;
        const int b = m / a.P, p = m - b * a.P;
        const float e[4] = {v.x, v.y, v.z, v.w};
        for (int j = 0; j < 4 && j < nv; ++j) {
          const int nn = n + j;
          const int slot = a.lay_cols > 0 ? nn / a.lay_cols : 0;
          const int nl = nn - slot * a.lay_cols;
          const int kv = nl / a.d_kv, rem = nl - kv * a.d_kv;
          const int g = rem / a.hd, cc = rem - g * a.hd;
          const size_t o = (size_t)slot * a.lay_stride + ((((size_t)kv * a.B + b) * G + g) * a.P + p) * a.hd + cc;
          reinterpret_cast<bf16_t*>(a.cache)[o] = f2bf(e[j]);
        }
      };
      epi_rows<RP, BN, CP, NT>(ct, rows, n0, N, f);
      break;
    }
    case EPI_EULER: {
      const CallParams* cp = a.cp;
      const float dt = cp->tau[a.step + 1] - cp->tau[a.step];
      auto f = [&](int r, int n, int nv, float4 v) {
        const int m = m0 + r;
        const int t = a.stok ? m % a.stok : 1;   // state-token rows: no action
        const int am = a.stok ? (m / a.stok) * (a.stok - 1) + t - 1 : m;
        if (t == 0) return;
        const float e[4] = {v.x, v.y, v.z, v.w};
        for (int j = 0; j < 4 && j < nv; ++j) {
          const int nn = n + j;
          const float vv = e[j] + a.bias[nn];
          float* ap = a.a + (size_t)am * N + nn;
          const float an = a.regression ? vv : (*ap + dt * vv);
          *ap = an;
          if (a.last) {
            float o = an;
            if (cp->act_std) o *= cp->act_std[nn];
            if (cp->act_mean) o += cp->act_mean[nn];
            cp->actions_out[(size_t)am * N + nn] = o;
          }
        }
      };
      epi_rows<RP, BN, CP, NT>(ct, rows, n0, N, f);
      break;
    }
    default:
      break;
  }
}

template <int MS, int NS>
__global__ __launch_bounds__(256) void gemm_tile_rs(GemmArgs a) {
  constexpr int BM = 32 * MS, BN = 32 * NS, ROWS = BM + BN;
  constexpr int LPT = ROWS * (TBK / 8) / 256;  // 16-byte loads per thread and slice
  constexpr int XL = BM / 32;                  // of which X rows
  static_assert(ROWS % 32 == 0 && LPT * 256 == ROWS * (TBK / 8), "tile rows");
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = a.M, N = a.N, K = a.K;
  // consecutive workgroups go to consecutive XCDs: unit u runs on XCD u / per
  const int per = gridDim.x >> 3;
  const int u = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  const int tiles = a.m_tiles * a.n_tiles;
  if (u >= tiles * a.nsplit) return;
  const int split = u / tiles, t = u - split * tiles;
  const int ntile = t / a.m_tiles, mtile = t - ntile * a.m_tiles;
  const int m0 = mtile * BM, n0 = ntile * BN;
  const int k0 = split * a.kper;
  const int k1 = min(K, k0 + a.kper);

  // this thread's rows: chunk ch of tile rows (tid >> 3) + 32 i
  const int ch = tid & 7;
  const bf16_t* src[LPT];
  bool rok[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int row = (tid >> 3) + 32 * i;
    if (i < XL) {
      const int m = m0 + row;
      rok[i] = m < M;
      src[i] = reinterpret_cast<const bf16_t*>(a.X) + (size_t)(rok[i] ? m : 0) * a.ldx + ch * 8;
    } else {
      const int n = n0 + row - BM;
      rok[i] = n < N;
      src[i] = reinterpret_cast<const bf16_t*>(a.W) + (size_t)(rok[i] ? n : 0) * K + ch * 8;
    }
  }
  uint4 pre[LPT];
  auto gload = [&](int kb) {
    const bool kok = kb + ch * 8 < k1;
#pragma unroll
    for (int i = 0; i < LPT; ++i) pre[i] = (rok[i] && kok) ? ldg16(src[i] + kb) : make_uint4(0, 0, 0, 0);
  };
  auto lstore = [&](int buf) {
    bf16_t* b = lds + (size_t)buf * ROWS * TPITCH;
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      *reinterpret_cast<uint4*>(b + ((tid >> 3) + 32 * i) * TPITCH + ch * 8) = pre[i];
  };

  f32x4 acc[MS][NS];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) acc[ms][ns] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(k0);
  lstore(0);
  __syncthreads();
  int buf = 0;
  for (int kb = k0; kb < k1; kb += TBK) {
    const bool more = kb + TBK < k1;
    if (more) gload(kb + TBK);
    const bf16_t* lb = lds + (size_t)buf * ROWS * TPITCH;
#pragma unroll
    for (int kk = 0; kk < TBK / 32; ++kk) {
      uint4 af[MS], bq[NS];
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        af[ms] = *reinterpret_cast<const uint4*>(lb + (wm * 16 * MS + ms * 16 + r16) * TPITCH + kk * 32 + g4 * 8);
#pragma unroll
      for (int ns = 0; ns < NS; ++ns)
        bq[ns] = *reinterpret_cast<const uint4*>(lb + (BM + wn * 16 * NS + ns * 16 + r16) * TPITCH + kk * 32 + g4 * 8);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) mma16(acc[ms][ns], af[ms], bq[ns], bf16_t());
    }
    if (more) lstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // Epilogue: the fp32 tile goes through LDS (the K-loop ended with a
  // barrier), then threads walk it row by row so that consecutive threads
  // finish consecutive columns.
  float* ct = reinterpret_cast<float*>(smem);  // [BM][CP]
  constexpr int CP = BN + 4;
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        ct[(wm * 16 * MS + ms * 16 + g4 * 4 + i) * CP + wn * 16 * NS + ns * 16 + r16] = acc[ms][ns][i];
  __syncthreads();
  tile_epilogue<BM, BN, CP>(a, ct, m0, n0, split);
}


// ---------------------------------------------------------------------------
// gemm_tile: the K-slices stream into a ring of NST LDS stages with
// direct-to-LDS loads (global_load_lds_dwordx4), NST - 1 slices ahead of the
// MFMAs, so several slices' latency overlaps without holding their bytes in
// registers.  A stage holds ROWS rows of 64 k-values (128 bytes); a load
// instruction of a wave fills 1 KB (eight rows), lane l writing row l/8,
// 16-byte slot l%8, and fetching the row's k-chunk (l%8) ^ (row%8): the XOR
// swizzle puts the eight rows one MFMA operand load reads into eight
// different bank groups.  Stages are separate LDS arrays indexed at compile
// time, so the compiler can tell the stage being read from the ones still in
// flight and does not wait for those.  Requires K % 64 == 0 (rows beyond M
// or N are loaded from a valid row and never stored).
//
// NWV waves: 4 in 2 x 2, or 8 in 2 x 4 (two per SIMD).  Every wave sums its
// outputs' k-products slice by slice in the same order, so the wave layout
// does not change a result.  The 256 x 256 tile (eight waves, 128 x 64 per
// wave) feeds 128 FLOP per staged byte instead of 85 (256 x 128); its two
// 64 KB stages fill the LDS, and a slice's MFMAs cover the next slice's load.
template <int MS, int NS, int NWV = 4>
struct Ring {
  static constexpr int BM = 32 * MS, BN = 32 * NS, ROWS = BM + BN;
  static constexpr int NST = ROWS <= 256 ? 4 : (ROWS <= 384 ? 3 : 2);   // stages (LDS <= 144 KB)
  static constexpr int LPT = ROWS * 8 / (64 * NWV);     // load instructions per thread and slice
  static constexpr int SB = ROWS * 8;                   // 16-byte slots per stage
  // rows of the fp32 output tile per epilogue pass (the tile goes through stage 0)
  static constexpr int RP = (64 * (BN + 4) * 4 <= SB * 16) ? 64 : (32 * (BN + 4) * 4 <= SB * 16 ? 32 : 16);
};

template <int MS, int NS, int NWV = 4>
__global__ __launch_bounds__(64 * NWV) void gemm_tile(GemmArgs a) {
  using R = Ring<MS, NS, NWV>;
  constexpr int BM = R::BM, BN = R::BN, NST = R::NST, LPT = R::LPT, SB = R::SB, D = NST - 1;
  constexpr int WN = NWV / 2;                          // waves along N (2 along M)
  constexpr int MSW = BM / 32, NSW = BN / (16 * WN);   // 16-row / 16-column subtiles of a wave
  constexpr int KKB = NWV == 8 ? 1 : 2;                // k-halves whose operands are read at once
  static_assert(LPT * 64 * NWV == R::ROWS * 8, "tile rows");
  __shared__ v4u st0[SB], st1[SB], st2[NST > 2 ? SB : 1], st3[NST > 3 ? SB : 1];
  auto stage = [&](auto j) -> v4u* {
    constexpr int J = decltype(j)::value;
    if constexpr (J == 0) return st0;
    else if constexpr (J == 1) return st1;
    else if constexpr (J == 2) return st2;
    else return st3;
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int M = a.M, N = a.N, K = a.K;
  const int per = gridDim.x >> 3;
  const int u = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  const int tiles = a.m_tiles * a.n_tiles;
  if (u >= tiles * a.nsplit) return;
  const int split = u / tiles, t = u - split * tiles;
  const int ntile = t / a.m_tiles, mtile = t - ntile * a.m_tiles;
  const int m0 = mtile * BM, n0 = ntile * BN;
  const int k0 = split * a.kper;
  const int nsl = (min(K, k0 + a.kper) - k0) / 64;

  // source of this lane's slot in load instruction i: row (i*NWV + wave)*8 + lane/8
  const bf16_t* src[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int row = (i * NWV + wave) * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ (row & 7);
    if (row < BM) {
      const int m = min(m0 + row, M - 1);
      src[i] = reinterpret_cast<const bf16_t*>(a.X) + (size_t)m * a.ldx + k0 + chunk * 8;
    } else {
      const int n = min(n0 + row - BM, N - 1);
      src[i] = reinterpret_cast<const bf16_t*>(a.W) + (size_t)n * K + k0 + chunk * 8;
    }
  }
  auto issue = [&](auto j, int sl) {
    v4u* b = stage(j);
#pragma unroll
    for (int i = 0; i < LPT; ++i) dma16(src[i] + sl * 64, b + (i * NWV + wave) * 64);
  };

  f32x4 acc[MSW][NSW];
#pragma unroll
  for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
    for (int ns = 0; ns < NSW; ++ns) acc[ms][ns] = f32x4{0.f, 0.f, 0.f, 0.f};

  // operand rows of this lane and their swizzled slot for logical chunk c.
  // With four waves every fragment of the slice is read before the first
  // MFMA, so the LDS latency of the second k-half hides behind the first
  // half's MFMAs; with eight the other wave of the SIMD hides it, and one
  // k-half at a time keeps the registers under the two-wave limit.
  auto compute = [&](const v4u* b) {
#pragma unroll
    for (int k2 = 0; k2 < 2; k2 += KKB) {
      v4u af[KKB][MSW], bq[KKB][NSW];
#pragma unroll
      for (int kq = 0; kq < KKB; ++kq) {
        const int c = (k2 + kq) * 4 + g4;
#pragma unroll
        for (int ms = 0; ms < MSW; ++ms) {
          const int row = wm * 16 * MSW + ms * 16 + r16;
          af[kq][ms] = b[row * 8 + (c ^ (row & 7))];
        }
#pragma unroll
        for (int ns = 0; ns < NSW; ++ns) {
          const int row = BM + wn * 16 * NSW + ns * 16 + r16;
          bq[kq][ns] = b[row * 8 + (c ^ (row & 7))];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kq = 0; kq < KKB; ++kq)
#pragma unroll
        for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
          for (int ns = 0; ns < NSW; ++ns)
            acc[ms][ns] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[kq][ms]),
                                                                  __builtin_bit_cast(bf16x8_t, bq[kq][ns]), acc[ms][ns],
                                                                  0, 0, 0);
    }
  };

  // prologue: slices 0 .. D-1 in flight
  [&]<int... J>(std::integer_sequence<int, J...>) {
    ((J < nsl ? issue(std::integral_constant<int, J>{}, J) : void()), ...);
  }(std::make_integer_sequence<int, D>{});

  for (int it0 = 0; it0 < nsl; it0 += NST) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      (
          [&] {
            const int it = it0 + J;
            if (it >= nsl) return;
            // slice `it` has landed once at most the D-1 later slices are pending
            if (it + D - 1 < nsl)
              __builtin_amdgcn_s_waitcnt(vm_wait((D - 1) * LPT));
            else
              __builtin_amdgcn_s_waitcnt(vm_wait(0));
            lds_barrier();
            // the stage of slice it-1 is free: refill it with slice it+D
            if (it + D < nsl) issue(std::integral_constant<int, (J + D) % NST>{}, it + D);
            compute(stage(std::integral_constant<int, J>{}));
          }(),
          ...);
    }(std::make_integer_sequence<int, NST>{});
  }
  __builtin_amdgcn_s_waitcnt(vm_wait(0));
  lds_barrier();

  // epilogue in passes of RP rows through stage 0
  constexpr int RP = R::RP, CP = BN + 4;
  float* ct = reinterpret_cast<float*>(st0);
#pragma unroll
  for (int p = 0; p < BM / RP; ++p) {
#pragma unroll
    for (int ms = 0; ms < MSW; ++ms) {
      const int rb = wm * 16 * MSW + ms * 16;  // first row of subtile ms
      if (rb / RP == p) {
#pragma unroll
        for (int ns = 0; ns < NSW; ++ns)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            ct[(rb - p * RP + g4 * 4 + i) * CP + wn * 16 * NSW + ns * 16 + r16] = acc[ms][ns][i];
      }
    }
    lds_barrier();  // LDS only: the epilogue's global stores need not complete here
    tile_epilogue<RP, BN, CP, 64 * NWV>(a, ct, m0 + p * RP, n0, split);
    lds_barrier();
  }
}

// ---------------------------------------------------------------------------
template <typename K_>
hipError_t set_lds_attr(K_ kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             160 * 1024);
}

template <typename T, int MS, int NSUB, int CPW>
hipError_t launch_skinny_t(const GemmArgs& a, int units, size_t lds, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = set_lds_attr(&gemm_skinny<T, MS, NSUB, CPW>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL((gemm_skinny<T, MS, NSUB, CPW>), dim3(units), dim3(64 * WKS), lds, s, a);
  return hipGetLastError();
}

template <typename T, int MS, int NSUB>
hipError_t skinny_cpw(int cpw, const GemmArgs& a, int units, size_t lds, hipStream_t s) {
  return cpw == 2 ? launch_skinny_t<T, MS, NSUB, 2>(a, units, lds, s) : launch_skinny_t<T, MS, NSUB, 1>(a, units, lds, s);
}

template <typename T>
hipError_t skinny_t(const SkinnyShape& sh, const GemmArgs& a, hipStream_t s) {
  switch (sh.ms * 10 + sh.nsub) {
    case 11: return skinny_cpw<T, 1, 1>(sh.cpw, a, sh.units, sh.lds, s);
    case 12: return skinny_cpw<T, 1, 2>(sh.cpw, a, sh.units, sh.lds, s);
    case 21: return skinny_cpw<T, 2, 1>(sh.cpw, a, sh.units, sh.lds, s);
    case 22: return skinny_cpw<T, 2, 2>(sh.cpw, a, sh.units, sh.lds, s);
    case 41: return skinny_cpw<T, 4, 1>(sh.cpw, a, sh.units, sh.lds, s);
    case 42: return skinny_cpw<T, 4, 2>(sh.cpw, a, sh.units, sh.lds, s);
    case 24: return launch_skinny_t<T, 2, 4, 1>(a, sh.units, sh.lds, s);
    case 44: return launch_skinny_t<T, 4, 4, 1>(a, sh.units, sh.lds, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int MS, int NSUB, int NC>
hipError_t launch_wide_t(const GemmArgs& a, int units, size_t lds, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = set_lds_attr(&gemm_wide<T, MS, NSUB, NC>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL((gemm_wide<T, MS, NSUB, NC>), dim3(units), dim3(256), lds, s, a);
  return hipGetLastError();
}

template <typename T, int MS, int NSUB>
hipError_t wide_nc(int nc, const GemmArgs& a, int units, size_t lds, hipStream_t s) {
  switch (nc) {
    case 1: return launch_wide_t<T, MS, NSUB, 1>(a, units, lds, s);
    case 2: return launch_wide_t<T, MS, NSUB, 2>(a, units, lds, s);
    case 4: return launch_wide_t<T, MS, NSUB, 4>(a, units, lds, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t wide_t(const WideShape& sh, const GemmArgs& a, hipStream_t s) {
  switch (sh.ms * 10 + sh.nsub) {
    case 11: return wide_nc<T, 1, 1>(sh.nc, a, sh.units, sh.lds, s);
    case 21: return wide_nc<T, 2, 1>(sh.nc, a, sh.units, sh.lds, s);
    case 41: return wide_nc<T, 4, 1>(sh.nc, a, sh.units, sh.lds, s);
    case 42: return wide_nc<T, 4, 2>(sh.nc, a, sh.units, sh.lds, s);
  }
  return hipErrorInvalidValue;
}


// K % 64 == 0: the direct-to-LDS ring on eight waves (two per SIMD, so one
// wave's LDS and load waits hide behind the other's MFMAs: 12-17% faster than
// four waves on every tile); else the register-staged kernel on four.
template <int MS, int NS>
hipError_t launch_tile_t(const TileShape& sh, const GemmArgs& a, hipStream_t s) {
  if (a.K % 64 == 0) {
    hipLaunchKernelGGL((gemm_tile<MS, NS, 8>), dim3(sh.grid), dim3(512), 0, s, a);
    return hipGetLastError();
  }
  if constexpr (MS * NS > 32) {   // 256 x 256: the ring only
    return hipErrorInvalidValue;
  } else {
    static bool attr = false;
    if (!attr) {
      hipError_t e = set_lds_attr(&gemm_tile_rs<MS, NS>);
      if (e != hipSuccess) return e;
      attr = true;
    }
    const size_t lds = tile_lds_bytes<MS, NS>();
    hipLaunchKernelGGL((gemm_tile_rs<MS, NS>), dim3(sh.grid), dim3(256), lds, s, a);
    return hipGetLastError();
  }
}

// The tiles gemm_tile is instantiated for, as (MS, NS), with the measured
// time of one 64-wide K-slice of a workgroup on eight waves (microseconds, one
// workgroup per compute unit: bound by the operand bytes a compute unit takes
// in from L2) and the fixed cost of a workgroup (pipeline fill, epilogue).
struct TileCand { int ms, ns; double slice_us, fixed_us; };
constexpr int kNumTiles = 5;
constexpr TileCand kTiles[kNumTiles] = {{2, 4, 0.34, 4.0}, {4, 4, 0.47, 5.0}, {8, 4, 0.80, 6.0}, {4, 8, 0.80, 6.0},
                                        {8, 8, 1.6, 8.0}};   // 256 x 256: K % 64 == 0 only

int cdiv_i(int a, int b) { return (a + b - 1) / b; }

}  // namespace

int gemm_chunk_k(int et) { return et == ET_BF16 ? 128 : 64; }

bool skinny_plan(int et, int M, int N, int K, int nsub, bool allow_split, SkinnyShape* sh) {
  const int KC = gemm_chunk_k(et);
  if (M > 128) return false;
  // Split-K partial outputs take any number of W subtiles: above 16 token rows
  // four subtiles per workgroup read each X row block for 64 W rows instead
  // of 16, which cuts the per-CU ingest that bounds these shapes -- as long as
  // the grid still fills the chip.
  if (nsub == 1 && allow_split && M > 16) {
    if (skinny_plan(et, M, N, K, 4, true, sh) && sh->units >= 192) return true;
  }
  // Gate/up pairs (no split): two pairs per workgroup above 64 token rows.
  if (nsub == 2 && M > 64) {
    if (skinny_plan(et, M, N, K, 4, false, sh) && sh->units >= 192) return true;
  }
  sh->ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  sh->nsub = nsub;
  sh->n_tiles = cdiv_i(N, 16 * nsub);
  sh->m_tiles = cdiv_i(M, 16 * sh->ms);
  const int chunks = cdiv_i(K, KC);
  const int base = sh->n_tiles * sh->m_tiles;
  // Split K only where the epilogue allows it, as far as keeps the grid in one
  // pass over the 256 compute units.
  int nsplit = 1;
  if (allow_split) nsplit = std::max(1, std::min(chunks, 256 / std::max(1, base)));
  // wide tiles: at least half the waves of a workgroup hold a chunk
  if (nsub == 4) nsplit = std::max(1, std::min(nsplit, chunks / (WKS / 2)));
  const int cps = cdiv_i(chunks, nsplit);  // chunks per split
  sh->nsplit = cdiv_i(chunks, cps);
  sh->kper = cps * KC;
  // two chunks per wave and round when the registers allow it
  sh->cpw = (cps > WKS && (sh->ms + nsub) * 2 * 16 + sh->ms * nsub * 4 <= 200) ? 2 : 1;
  sh->units = base * sh->nsplit;
  sh->lds = (size_t)WKS * sh->ms * nsub * 64 * 16;
  return true;
}

void wide_plan(int et, int M, int N, int K, int nsub, WideShape* sh) {
  const int es = et == ET_BF16 ? 2 : 4;
  const int E = 16 / es;
  const int KC = gemm_chunk_k(et);
  sh->ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  if (nsub == 2) sh->ms = 4;
  sh->nsub = nsub;
  sh->nc = K <= KC ? 1 : (K <= 2 * KC ? 2 : 4);
  const int MT = 16 * sh->ms;
  sh->n_tiles = cdiv_i(N, 64 * nsub);
  sh->m_tiles = cdiv_i(M, MT);
  sh->units = sh->n_tiles * sh->m_tiles;
  sh->lds = (size_t)MT * (sh->nc * KC + E) * es;
}

hipError_t launch_gemm_skinny(int et, const SkinnyShape& sh, GemmArgs a, hipStream_t s) {
  if (sh.units <= 0) return hipSuccess;
  a.n_tiles = sh.n_tiles;
  a.nsplit = sh.nsplit;
  a.kper = sh.kper;
  return et == ET_BF16 ? skinny_t<bf16_t>(sh, a, s) : skinny_t<float>(sh, a, s);
}

hipError_t launch_gemm_wide(int et, const WideShape& sh, GemmArgs a, hipStream_t s) {
  if (sh.units <= 0) return hipSuccess;
  a.n_tiles = sh.n_tiles;
  a.nsplit = 1;
  return et == ET_BF16 ? wide_t<bf16_t>(sh, a, s) : wide_t<float>(sh, a, s);
}

bool tile_plan(int et, int M, int N, int K, bool allow_split, int force, TileShape* sh) {
  if (et != ET_BF16 || M <= 128 || K % 8 || force >= kNumTiles) return false;
  const int slices = cdiv_i(K, TBK);
  double best = 1e30;
  for (int c = 0; c < kNumTiles; ++c) {
    if (force >= 0 && c != force) continue;
    const TileCand& tc = kTiles[c];
    if (tc.ms * tc.ns > 32 && K % 64) continue;   // the eight-wave tile runs on the direct-to-LDS ring only
    const int BM = 32 * tc.ms, BN = 32 * tc.ns;
    const int mt = cdiv_i(M, BM), nt = cdiv_i(N, BN);
    const int max_split = (allow_split && force < 0) ? std::min(8, slices) : 1;
    for (int ns = 1; ns <= max_split; ++ns) {
      const int sps = cdiv_i(slices, ns);  // slices per split
      const int nsplit = cdiv_i(slices, sps);
      if (ns > 1 && nsplit != ns) continue;
      const int units = mt * nt * nsplit;
      const double rounds = std::ceil(units / 256.0);
      const double unit_us = tc.fixed_us + sps * tc.slice_us;
      // split partials: written once, read once more by the row kernel
      const double split_us = nsplit > 1 ? 8.0 * M * N * nsplit / 4.0e6 : 0.0;
      const double cost = rounds * unit_us + split_us;
      if (cost < best) {
        best = cost;
        sh->ms = tc.ms; sh->ns = tc.ns; sh->nsplit = nsplit; sh->kper = sps * TBK;
        sh->m_tiles = mt; sh->n_tiles = nt; sh->units = units; sh->grid = cdiv_i(units, 8) * 8;
      }
    }
  }
  if (best >= 1e30) return false;
  switch (sh->ms * 10 + sh->ns) {
    case 24: sh->lds = tile_lds_bytes<2, 4>(); break;
    case 44: sh->lds = tile_lds_bytes<4, 4>(); break;
    case 84: sh->lds = tile_lds_bytes<8, 4>(); break;
    case 48: sh->lds = tile_lds_bytes<4, 8>(); break;
    default: sh->lds = 0; break;   // 256 x 256: static LDS only
  }
  return true;
}

hipError_t launch_gemm_tile(const TileShape& sh, GemmArgs a, hipStream_t s) {
  if (sh.units <= 0) return hipSuccess;
  a.n_tiles = sh.n_tiles;
  a.m_tiles = sh.m_tiles;
  a.nsplit = sh.nsplit;
  a.kper = sh.kper;
  switch (sh.ms * 10 + sh.ns) {
    case 24: return launch_tile_t<2, 4>(sh, a, s);
    case 44: return launch_tile_t<4, 4>(sh, a, s);
    case 84: return launch_tile_t<8, 4>(sh, a, s);
    case 48: return launch_tile_t<4, 8>(sh, a, s);
    case 88: return launch_tile_t<8, 8>(sh, a, s);
  }
  return hipErrorInvalidValue;
}

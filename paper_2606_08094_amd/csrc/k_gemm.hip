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
// gemm_wide -- large M (prefix K/V build, batched requests).  Four waves along
//   N (NT = 64*NSUB), X staged per K-slice in LDS and shared by the four
//   waves, K-slices looped inside the workgroup.
//
// Operand layout: in a chunk, lane l of a wave reads 16-byte vector v of row
// (l % 16) at k-offset v*4*E + (l/16)*E, for W and X alike, so the MFMA's k
// order is a permutation common to both operands and every load instruction
// of a wave reads 64 contiguous bytes per row.
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

int cdiv_i(int a, int b) { return (a + b - 1) / b; }

}  // namespace

int gemm_chunk_k(int et) { return et == ET_BF16 ? 128 : 64; }

bool skinny_plan(int et, int M, int N, int K, int nsub, bool allow_split, SkinnyShape* sh) {
  const int KC = gemm_chunk_k(et);
  if (M > 128) return false;
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

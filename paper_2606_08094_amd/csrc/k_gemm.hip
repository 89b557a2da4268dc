// MFMA GEMMs y = X W^T for the expert's projections.  No workgroup ever
// waits on another: an output tile is reduced inside one workgroup, or written
// as a split-K partial that a later launch adds up (on this 8-XCD part an
// agent-scope fence writes back and invalidates the XCD's whole L2, so
// in-kernel cross-workgroup reductions cost far more than a launch).
//
// gemm_skinny -- the per-step projections, M <= 128 token rows.
//   A workgroup of 8 waves owns 16*NSUB rows of W (NSUB = 2: a gate/up pair
//   of interleaved 16-row blocks) and a K-range of up to 8*CPW chunks of
//   KC = 4*VPL*E k-values (split-K across workgroups when K is longer).  Every
//   wave first issues the loads of its W chunks (the HBM stream), then the
//   workgroup stages the [MT][K-range] X tile in LDS with all of a thread's
//   loads in flight at once; wave w multiplies chunks w, w+8, ...  The eight
//   partial tiles are summed in wave order through LDS and wave 0 runs the
//   epilogue.
//
// gemm_wide -- large M or very large N (prefix K/V build, modulation tables,
//   batched requests).  Four waves along N (NT = 64*NSUB), X staged per K-slice
//   in LDS and shared by the four waves, K-slices looped inside the workgroup.
//
// In both, lane l of a wave loads 64 contiguous bytes of W row (l % 16) at
// k-offset (l / 16) * KCL of a chunk, and reads X with the same k mapping, so
// the MFMA's k order is a permutation common to both operands.
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
  constexpr int KCL = VPL * E;
  constexpr int KC = 4 * KCL;
  constexpr int MT = 16 * MS;
  extern __shared__ __align__(16) unsigned char smem[];
  T* xs = reinterpret_cast<T*>(smem);               // [MT][pitch]
  f32x4* red = reinterpret_cast<f32x4*>(smem);      // reuses the X tile after the MFMA loop

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int N = a.N, K = a.K;
  int bid = blockIdx.x;
  const int split = bid % a.nsplit;
  bid /= a.nsplit;
  const int ntile = bid % a.n_tiles, mtile = bid / a.n_tiles;
  const int m0 = mtile * MT;
  const int nb = ntile * 16 * NSUB;
  const int k0 = split * (WKS * CPW * KC);
  const int k1 = min(K, k0 + WKS * CPW * KC);
  const int nck = (k1 - k0 + KC - 1) / KC;
  const int pitch = nck * KC + E;

  // 1. W chunks of this wave -> registers
  const T* W = reinterpret_cast<const T*>(a.W);
  uint4 wreg[CPW][NSUB][VPL];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int kc = k0 + (wave + j * WKS) * KC + g4 * KCL;
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int n = nb + s * 16 + r16;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int k = kc + v * E;
        wreg[j][s][v] = (n < N && k < k1) ? ldg16(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
      }
    }
  }

  // 2. the X tile of this K-range in LDS
  stage_x<T, MT>(a, xs, pitch, m0, k0, nck * KC);
  __syncthreads();

  // 3. MFMA over this wave's chunks
  f32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int c = wave + j * WKS;
    if (c >= nck) break;
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) {
      const T* xrow = xs + (size_t)(ms * 16 + r16) * pitch + c * KC + g4 * KCL;
      uint4 xf[VPL];
#pragma unroll
      for (int v = 0; v < VPL; ++v) xf[v] = *reinterpret_cast<const uint4*>(xrow + v * E);
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
#pragma unroll
        for (int v = 0; v < VPL; ++v) mma16(acc[ms][s], xf[v], wreg[j][s][v], T());
    }
  }

  // 4. sum the eight partial tiles in wave order; epilogue on wave 0
  __syncthreads();  // every wave is done reading the X tile
  if (wave > 0) {
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int s = 0; s < NSUB; ++s) red[(((wave - 1) * MS + ms) * NSUB + s) * 64 + lane] = acc[ms][s];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 1; w < WKS; ++w)
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int s = 0; s < NSUB; ++s) acc[ms][s] += red[(((w - 1) * MS + ms) * NSUB + s) * 64 + lane];
  wave_epilogue<T, MS, NSUB>(a, acc, m0, nb, split);
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
  const int es = et == ET_BF16 ? 2 : 4;
  const int E = 16 / es;
  const int KC = gemm_chunk_k(et);
  if (M > 128) return false;
  sh->ms = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int MT = 16 * sh->ms;
  sh->nsub = nsub;
  // K-range per workgroup: 8 or 16 chunks, as long as the X tile fits in LDS
  sh->cpw = ((size_t)MT * (2 * WKS * KC + E) * es <= 136 * 1024) ? 2 : 1;
  const int krange = WKS * sh->cpw * KC;
  sh->nsplit = cdiv_i(K, krange);
  if (sh->nsplit > 1 && !allow_split) return false;
  if (sh->nsplit == 1 && sh->cpw == 2 && K <= WKS * KC) sh->cpw = 1;
  sh->n_tiles = cdiv_i(N, 16 * nsub);
  sh->m_tiles = cdiv_i(M, MT);
  sh->units = sh->n_tiles * sh->m_tiles * sh->nsplit;
  const int kr = std::min(K, WKS * sh->cpw * KC);
  const size_t tile = (size_t)MT * (cdiv_i(kr, KC) * KC + E) * es;
  const size_t red = (size_t)(WKS - 1) * sh->ms * nsub * 64 * 16;
  sh->lds = std::max(tile, red);
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
  return et == ET_BF16 ? skinny_t<bf16_t>(sh, a, s) : skinny_t<float>(sh, a, s);
}

hipError_t launch_gemm_wide(int et, const WideShape& sh, GemmArgs a, hipStream_t s) {
  if (sh.units <= 0) return hipSuccess;
  a.n_tiles = sh.n_tiles;
  a.nsplit = 1;
  return et == ET_BF16 ? wide_t<bf16_t>(sh, a, s) : wide_t<float>(sh, a, s);
}

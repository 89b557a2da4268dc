// Skinny MFMA GEMM y = X W^T for the expert's projections (M = chunk tokens).
//
// One workgroup (4 waves) owns a tile of MT = 16*MS rows of X, NT = 64*NSUB
// rows of W and one K-slice of KS = NC*KC columns.  Each wave owns 16*NSUB rows
// of W: it issues the loads of its whole K-slice into registers first (they
// are the HBM stream; nothing else is waited on before they are in flight),
// then the workgroup stages its X slice once in LDS, applying the adaRMS
// prologue on the way, and every wave multiplies its W rows against all MT
// rows of X.  Lane l of a wave loads 64 contiguous bytes of W row (l % 16) at
// k-offset (l / 16) * KCL of each chunk; X fragments are read from LDS with
// the same k mapping, so the MFMA's k order is a permutation shared by both
// operands and the result is unchanged.
//
// Split-K partials go to a workspace; the last workgroup to arrive on a tile
// sums them in split order (deterministic) and runs the epilogue.
#include "gemm_epilogue.h"

namespace {

template <typename T, int MS, int NSUB, int NC>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int VPL = 4;
  constexpr int KCL = VPL * E;
  constexpr int KC = 4 * KCL;
  constexpr int KS = NC * KC;
  constexpr int MT = 16 * MS;
  constexpr int NT = 64 * NSUB;
  constexpr int PITCH = KS + E;  // LDS row pitch in elements (16-byte pad)

  extern __shared__ __align__(16) unsigned char smem[];
  T* xs = reinterpret_cast<T*>(smem);
  float* rstd_s = reinterpret_cast<float*>(smem + (size_t)MT * PITCH * sizeof(T));
  float* red_s = rstd_s + MT;          // [4][MT]
  int* flag_s = reinterpret_cast<int*>(red_s + 4 * MT);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;

  int unit = blockIdx.x;
  const int split = unit % a.nsplit;
  unit /= a.nsplit;
  const int ntile = unit % a.n_tiles;
  const int mtile = unit / a.n_tiles;
  const int m0 = mtile * MT;
  const int k0 = split * KS;
  const int kend = min(K, k0 + KS);
  const int nw0 = ntile * NT + wave * 16 * NSUB;

  // 1. The W slice of this wave, straight to registers.
  const T* W = reinterpret_cast<const T*>(a.W);
  uint4 wreg[NSUB][NC][VPL];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    const int n = nw0 + s * 16 + r16;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int k = k0 + c * KC + g4 * KCL + v * E;
        wreg[s][c][v] = (n < N && k < kend) ? ldg16(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
      }
  }

  // 2. X slice -> LDS (adaRMS applied on the fly).
  if (a.rowss != nullptr) {
    if (tid < MT) {
      const int m = m0 + tid;
      float r = 0.0f;
      if (m < M) {
        float ss = 0.0f;
        for (int p = 0; p < a.rowss_np; ++p) ss += a.rowss[(size_t)p * M + m];
        r = 1.0f / sqrtf(ss / (float)K + a.eps);
      }
      rstd_s[tid] = r;
    }
    __syncthreads();
  }
  constexpr int VROW = KS / E;
  for (int i = tid; i < MT * VROW; i += 256) {
    const int row = i / VROW, kv = i - row * VROW;
    const int m = m0 + row, k = k0 + kv * E;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (m < M && k < kend) {
      if (a.rowss == nullptr) {
        val = ldg16(reinterpret_cast<const T*>(a.X) + (size_t)m * a.ldx + k);
      } else {
        const float* xr = reinterpret_cast<const float*>(a.X) + (size_t)m * a.ldx + k;
        float u[E];
        const float rs = rstd_s[row];
#pragma unroll
        for (int e = 0; e < E; e += 4) {
          const float4 xv = *reinterpret_cast<const float4*>(xr + e);
          const float4 gv = *reinterpret_cast<const float4*>(a.gamma + k + e);
          const float4 bv = *reinterpret_cast<const float4*>(a.beta + k + e);
          u[e + 0] = xv.x * rs * (1.0f + gv.x) + bv.x;
          u[e + 1] = xv.y * rs * (1.0f + gv.y) + bv.y;
          u[e + 2] = xv.z * rs * (1.0f + gv.z) + bv.z;
          u[e + 3] = xv.w * rs * (1.0f + gv.w) + bv.w;
        }
        val = pack16(u, T());
      }
    }
    stg16(xs + (size_t)row * PITCH + kv * E, val);
  }
  __syncthreads();

  // 3. MFMA over the slice.
  f32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (k0 + c * KC >= kend) break;
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) {
      uint4 xf[VPL];
      const T* xrow = xs + (size_t)(ms * 16 + r16) * PITCH + c * KC + g4 * KCL;
#pragma unroll
      for (int v = 0; v < VPL; ++v) xf[v] = *reinterpret_cast<const uint4*>(xrow + v * E);
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
#pragma unroll
        for (int v = 0; v < VPL; ++v) mma16(acc[ms][s], xf[v], wreg[s][c][v], T());
    }
  }

  // 4. Split-K: partials to the workspace, the last arrival reduces.
  if (a.nsplit > 1) {
    const int tile = mtile * a.n_tiles + ntile;
    constexpr int PER = 4 * MS * NSUB * 64;  // f32x4 per (tile, split)
    f32x4* wsp = reinterpret_cast<f32x4*>(a.ws) + ((size_t)tile * a.nsplit) * PER;
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
        wsp[(size_t)split * PER + ((wave * MS + ms) * NSUB + s) * 64 + lane] = acc[ms][s];
    if (!splitk_arrive_last(&a.cnt[tile], (unsigned)a.nsplit, flag_s)) return;
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        f32x4 t = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int sp = 0; sp < a.nsplit; ++sp) {
          t += wsp[(size_t)sp * PER + ((wave * MS + ms) * NSUB + s) * 64 + lane];
        }
        acc[ms][s] = t;
      }
  }

  gemm_epilogue<T, MS, NSUB>(a, acc, m0, ntile, nw0, red_s);
}

template <typename T, int MS, int NSUB, int NC>
hipError_t launch_one(const GemmArgs& a, int units, hipStream_t s) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int KS = NC * 16 * E;
  constexpr int MT = 16 * MS;
  const size_t lds = (size_t)MT * (KS + E) * sizeof(T) + (size_t)(MT + 4 * MT) * 4 + 16;
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, MS, NSUB, NC>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_done = true;
  }
  hipLaunchKernelGGL((gemm_kernel<T, MS, NSUB, NC>), dim3(units), dim3(256), lds, s, a);
  return hipGetLastError();
}

template <typename T, int MS, int NSUB>
hipError_t dispatch_nc(int nc, const GemmArgs& a, int units, hipStream_t s) {
  switch (nc) {
    case 1: return launch_one<T, MS, NSUB, 1>(a, units, s);
    case 2: return launch_one<T, MS, NSUB, 2>(a, units, s);
    case 4: return launch_one<T, MS, NSUB, 4>(a, units, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int MS>
hipError_t dispatch_nsub(int nsub, int nc, const GemmArgs& a, int units, hipStream_t s) {
  return nsub == 2 ? dispatch_nc<T, MS, 2>(nc, a, units, s) : dispatch_nc<T, MS, 1>(nc, a, units, s);
}

template <typename T>
hipError_t dispatch_ms(int ms, int nsub, int nc, const GemmArgs& a, int units, hipStream_t s) {
  switch (ms) {
    case 1: return dispatch_nsub<T, 1>(nsub, nc, a, units, s);
    case 2: return dispatch_nsub<T, 2>(nsub, nc, a, units, s);
    case 4: return dispatch_nsub<T, 4>(nsub, nc, a, units, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int gemm_chunk_k(int et) { return et == ET_BF16 ? 128 : 64; }

size_t gemm_lds_bytes(int et, int ms, int nc) {
  const int E = et == ET_BF16 ? 8 : 4;
  const int esz = et == ET_BF16 ? 2 : 4;
  const int MT = 16 * ms, KS = nc * 16 * E;
  return (size_t)MT * (KS + E) * esz + (size_t)(5 * MT) * 4 + 16;
}

size_t gemm_ws_floats_per_unit(int ms, int nsub) { return (size_t)4 * ms * nsub * 64 * 4; }

hipError_t launch_gemm(int et, int ms, int nsub, int nc, const GemmArgs& a, int units, hipStream_t s) {
  if (units <= 0) return hipSuccess;
  return et == ET_BF16 ? dispatch_ms<bf16_t>(ms, nsub, nc, a, units, s)
                       : dispatch_ms<float>(ms, nsub, nc, a, units, s);
}

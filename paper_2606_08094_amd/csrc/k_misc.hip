// Small per-chunk and per-step kernels of the denoise loop: per-call
// parameters, chunk start, input embedding, solver-time embedding, the int8
// activation quantiser of the W2A8 path, and finite checks.
#include "device_common.h"

namespace {

__global__ void set_params_kernel(CallParams* dst, CallParams src) {
  if (threadIdx.x == 0) *dst = src;
}

// a <- noise; xs[b] = b_in + b_s + state[b] W_s^T (the per-request constant part
// of the input embedding).
template <typename T>
__global__ __launch_bounds__(256) void init_chunk_kernel(const CallParams* cp, float* a, float* xs,
                                                          const T* W_s, const float* b_s,
                                                          const float* b_in, int n, int A, int S, int d) {
  const int b = blockIdx.x;
  const float* st = cp->state + (size_t)b * S;
  for (int j = threadIdx.x; j < d; j += 256) {
    float acc = b_in[j] + b_s[j];
    for (int s = 0; s < S; ++s) acc += st[s] * ElemTraits<T>::to_f(W_s[(size_t)j * S + s]);
    xs[(size_t)b * d + j] = acc;
  }
  const float* nz = cp->noise + (size_t)b * n * A;
  for (int i = threadIdx.x; i < n * A; i += 256) a[(size_t)b * n * A + i] = nz[i];
}

// x[m] = a[m] W_in^T + xs[b] + E_pos[token]; rowss[p][m] = sum of x^2 over
// columns 64p .. 64p+63 (the same partition as the residual GEMM epilogue).
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const float* a, const T* W_in, const float* xs,
                                                     const T* E_pos, float* x, float* rowss, int M, int n,
                                                     int A, int d) {
  const int m = blockIdx.x;
  const int b = m / n, tok = m - b * n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ float arow[64];
  for (int i = threadIdx.x; i < A; i += 256) arow[i] = a[(size_t)m * A + i];
  __syncthreads();
  const int npart = (d + 63) / 64;
  for (int j0 = 0; j0 < d; j0 += 256) {
    const int j = j0 + threadIdx.x;
    float v = 0.0f;
    if (j < d) {
      v = xs[(size_t)b * d + j] + ElemTraits<T>::to_f(E_pos[(size_t)tok * d + j]);
      for (int k = 0; k < A; ++k) v += arow[k] * ElemTraits<T>::to_f(W_in[(size_t)j * A + k]);
      x[(size_t)m * d + j] = v;
    }
    const float ss = wave_sum(v * v);
    const int p = j0 / 64 + wave;
    if (lane == 0 && p < npart) rowss[(size_t)p * M + m] = ss;
  }
}

// e[k] = [sin(2 pi tau_k / p_j), cos(2 pi tau_k / p_j)], p_j geometric from
// 4e-3 to 4; rows T..Tpad-1 are zero.  The angle is formed in double precision.
template <typename T>
__global__ __launch_bounds__(256) void time_embed_kernel(const CallParams* cp, T* e, int T_, int d) {
  const int k = blockIdx.x;
  const int half = d / 2;
  for (int j = threadIdx.x; j < half; j += 256) {
    float sv = 0.0f, cv = 0.0f;
    if (k < T_) {
      const double frac = (double)j / (double)(half > 1 ? half - 1 : 1);
      const double period = 4e-3 * pow(1000.0, frac);
      const double ang = 2.0 * 3.14159265358979323846 * (double)cp->tau[k] / period;
      sv = (float)sin(ang);
      cv = (float)cos(ang);
    }
    e[(size_t)k * d + j] = ElemTraits<T>::from_f(sv);
    e[(size_t)k * d + j + half] = ElemTraits<T>::from_f(cv);
  }
}

__global__ void copy_f32_kernel(float* dst, const float* src, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ void fill_u32_kernel(unsigned* p, unsigned v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Per-token absmax int8 quantiser (IEEE fp32): r = max(max|u|, 1e-5),
// q = clamp(rne(u * (127 / r)), -128, 127), with a correctly rounded divide.
__global__ __launch_bounds__(256) void quantize_kernel(QuantArgs a) {
  extern __shared__ float us[];
  __shared__ float red[4];
  __shared__ float rstd_s;
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (a.adarms) {
    if (threadIdx.x == 0) {
      float ss = 0.0f;
      for (int p = 0; p < a.rowss_np; ++p) ss += a.rowss[(size_t)p * a.M + m];
      rstd_s = 1.0f / sqrtf(ss / (float)a.K + a.eps);
    }
    __syncthreads();
  }
  float amax = 0.0f;
  for (int k = threadIdx.x; k < a.K; k += 256) {
    float v;
    if (a.src_type == 1)
      v = bf2f(reinterpret_cast<const bf16_t*>(a.x)[(size_t)m * a.ldx + k]);
    else
      v = reinterpret_cast<const float*>(a.x)[(size_t)m * a.ldx + k];
    if (a.adarms) v = v * rstd_s * (1.0f + a.gamma[k]) + a.beta[k];
    us[k] = v;
    amax = fmaxf(amax, fabsf(v));
  }
  amax = wave_max(amax);
  if (lane == 0) red[wave] = amax;
  __syncthreads();
  const float r = fmaxf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])), 1e-5f);
  const float inv = __fdiv_rn(127.0f, r);
  for (int k = threadIdx.x; k < a.K; k += 256) {
    const float qv = rintf(__fmul_rn(us[k], inv));
    a.q[(size_t)m * a.K + k] = (int8_t)fminf(fmaxf(qv, -128.0f), 127.0f);
  }
  if (threadIdx.x == 0) a.r[m] = r;
}

__global__ void check_finite_kernel(const float* x, size_t n, int* flag) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    if (!isfinite(x[i])) atomicOr(flag, 1);
}

}  // namespace

hipError_t launch_set_params(CallParams* dst, const CallParams& src, hipStream_t s) {
  hipLaunchKernelGGL(set_params_kernel, dim3(1), dim3(64), 0, s, dst, src);
  return hipGetLastError();
}

hipError_t launch_init_chunk(int et, const CallParams* cp, float* a, float* xs, const void* W_s,
                             const float* b_s, const float* b_in, int B, int n, int A, int S, int d,
                             hipStream_t s) {
  if (et == ET_BF16)
    hipLaunchKernelGGL(init_chunk_kernel<bf16_t>, dim3(B), dim3(256), 0, s, cp, a, xs,
                       reinterpret_cast<const bf16_t*>(W_s), b_s, b_in, n, A, S, d);
  else
    hipLaunchKernelGGL(init_chunk_kernel<float>, dim3(B), dim3(256), 0, s, cp, a, xs,
                       reinterpret_cast<const float*>(W_s), b_s, b_in, n, A, S, d);
  return hipGetLastError();
}

hipError_t launch_embed(int et, const float* a, const void* W_in, const float* xs, const void* E_pos,
                        float* x, float* rowss, int B, int n, int A, int d, hipStream_t s) {
  const int M = B * n;
  if (et == ET_BF16)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(M), dim3(256), 0, s, a, reinterpret_cast<const bf16_t*>(W_in),
                       xs, reinterpret_cast<const bf16_t*>(E_pos), x, rowss, M, n, A, d);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, a, reinterpret_cast<const float*>(W_in),
                       xs, reinterpret_cast<const float*>(E_pos), x, rowss, M, n, A, d);
  return hipGetLastError();
}

hipError_t launch_time_embed(int et, const CallParams* cp, void* e, int T, int Tpad, int d, hipStream_t s) {
  if (et == ET_BF16)
    hipLaunchKernelGGL(time_embed_kernel<bf16_t>, dim3(Tpad), dim3(256), 0, s, cp,
                       reinterpret_cast<bf16_t*>(e), T, d);
  else
    hipLaunchKernelGGL(time_embed_kernel<float>, dim3(Tpad), dim3(256), 0, s, cp, reinterpret_cast<float*>(e),
                       T, d);
  return hipGetLastError();
}

hipError_t launch_copy_f32(float* dst, const float* src, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(copy_f32_kernel, dim3(blocks), dim3(256), 0, s, dst, src, n);
  return hipGetLastError();
}

hipError_t launch_fill_u32(unsigned* p, unsigned v, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(fill_u32_kernel, dim3(blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_kernel, dim3(a.M), dim3(256), (size_t)a.K * sizeof(float), s, a);
  return hipGetLastError();
}

hipError_t launch_check_finite(const float* x, size_t n, int* flag, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(check_finite_kernel, dim3(blocks), dim3(256), 0, s, x, n, flag);
  return hipGetLastError();
}

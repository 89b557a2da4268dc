// Small per-chunk and per-step kernels of the denoise loop: per-call
// parameters, chunk start, input embedding, solver-time embedding, the int8
// activation quantiser of the W2A8 path, and finite checks.
#include <cmath>
#include "device_common.h"

namespace {

__global__ void set_params_kernel(CallParams* dst, CallParams src) {
  if (threadIdx.x == 0) *dst = src;
}

// Chunk start, one launch: a <- noise; xs[b] = b_in + b_s + state[b] W_s^T
// (the per-request constant part of the input embedding); and, when e is set,
// the sinusoidal embedding of every solver time: e[k] = [sin(2 pi tau_k / p_j),
// cos(2 pi tau_k / p_j)], p_j geometric from 4e-3 to 4, with rows T..Tpad-1
// zero and the angle formed in double precision.  Workgroups [0, B * XB) take
// 64 columns of one request's xs each (four threads split the state sum) and
// a share of its noise copy; the next Tpad * EB take 256 frequency pairs of
// one time row each.
constexpr int XCOLS = 64;
template <typename T>
__global__ __launch_bounds__(256) void chunk_start_kernel(const CallParams* cp, float* a, float* xs,
                                                          const T* W_s, const float* b_s,
                                                          const float* b_in, int B, int n, int A, int S, int d,
                                                          T* e, int T_, int Tpad) {
  const int XB = (d + XCOLS - 1) / XCOLS;
  const int tid = threadIdx.x;
  int blk = blockIdx.x;
  if (blk < B * XB) {
    __shared__ float red[4][XCOLS];
    const int b = blk / XB, cb = blk - b * XB;
    const int c = tid % XCOLS, part = tid / XCOLS;
    const int j = cb * XCOLS + c;
    const float* st = cp->state + (size_t)b * S;
    float acc = 0.0f;
    if (j < d)
      for (int s2 = part; s2 < S; s2 += 4) acc += st[s2] * ElemTraits<T>::to_f(W_s[(size_t)j * S + s2]);
    red[part][c] = acc;
    __syncthreads();
    if (part == 0 && j < d)   // b_in NULL: the state token's own row
      xs[(size_t)b * d + j] = (b_in ? b_in[j] : 0.0f) + b_s[j] + red[0][c] + red[1][c] + red[2][c] + red[3][c];
    const float* nz = cp->noise + (size_t)b * n * A;
    const int per = (n * A + XB - 1) / XB;
    const int i1 = min(n * A, (cb + 1) * per);
    for (int i = cb * per + tid; i < i1; i += 256) a[(size_t)b * n * A + i] = nz[i];
    return;
  }
  blk -= B * XB;
  const int half = d / 2, EB = (half + 255) / 256;
  const int k = blk / EB, j = (blk - k * EB) * 256 + tid;
  if (e == nullptr || k >= Tpad || j >= half) return;
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

// One workgroup per token row: finish the residual stream x (add the split-K
// partials of a residual projection, form the input embedding, or take the
// backbone's input rows) and write the next sublayer's adaRMS input u.  A thread owns the columns
// 4*(tid + 256*i); all of its loads are issued before the row reduction.
template <typename T>
__global__ __launch_bounds__(256) void row_norm_kernel(RowNormArgs a) {
  constexpr int CPT = 4;  // float4 groups per thread: d <= 4 * 256 * CPT
  const int m = blockIdx.x;
  const int d = a.d;
  const int t = threadIdx.x;
  __shared__ float red[4];
  float4 xv[CPT];
  float ss = 0.0f;
  if (a.mode == 0) {
    const float* xr = a.x + (size_t)m * d;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = 4 * (t + 256 * i);
      xv[i] = c < d ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (a.alpha != nullptr) {
      float4 ps[CPT], al[CPT];
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int c = 4 * (t + 256 * i);
        ps[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        al[i] = c < d ? *reinterpret_cast<const float4*>(a.alpha + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      for (int s0 = 0; s0 < a.nsplit; s0 += 4) {
        float4 pv[4][CPT];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int i = 0; i < CPT; ++i) {
            const int c = 4 * (t + 256 * i);
            pv[u][i] = (s0 + u < a.nsplit && c < d)
                           ? *reinterpret_cast<const float4*>(a.part + ((size_t)(s0 + u) * a.M + m) * d + c)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
          }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int i = 0; i < CPT; ++i) {
            ps[i].x += pv[u][i].x; ps[i].y += pv[u][i].y; ps[i].z += pv[u][i].z; ps[i].w += pv[u][i].w;
          }
      }
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        xv[i].x += al[i].x * ps[i].x; xv[i].y += al[i].y * ps[i].y;
        xv[i].z += al[i].z * ps[i].z; xv[i].w += al[i].w * ps[i].w;
      }
    }
  } else if (a.mode == 2) {
    const T* xr = reinterpret_cast<const T*>(a.x_in) + (size_t)m * d;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = 4 * (t + 256 * i);
      xv[i] = c < d ? make_float4(ElemTraits<T>::to_f(xr[c]), ElemTraits<T>::to_f(xr[c + 1]),
                                  ElemTraits<T>::to_f(xr[c + 2]), ElemTraits<T>::to_f(xr[c + 3]))
                    : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  } else {
    const int b = m / a.n, tok = m - b * a.n;
    // state-token variant: row 0 of a request is the projected state alone
    const bool srow = a.stok && tok == 0;
    const int ai = a.stok ? b * (a.n - 1) + tok - 1 : m;   // action row
    const int et = a.stok ? tok - 1 : tok;                  // its E_pos row
    __shared__ float arow[64];
    if (t < a.A) arow[t] = srow ? 0.0f : a.a[(size_t)ai * a.A + t];
    __syncthreads();
    const T* W = reinterpret_cast<const T*>(a.W_in);
    const T* ep = reinterpret_cast<const T*>(a.E_pos) + (size_t)(srow ? 0 : et) * d;
    const float* base = a.stok && !srow ? a.b_in : a.xs + (size_t)b * d;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = 4 * (t + 256 * i);
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (c < d && srow) {
        const float4 x4 = *reinterpret_cast<const float4*>(base + c);
        v[0] = x4.x;
        v[1] = x4.y;
        v[2] = x4.z;
        v[3] = x4.w;
      } else if (c < d) {
        const float4 x4 = *reinterpret_cast<const float4*>(base + c);
        v[0] = x4.x + ElemTraits<T>::to_f(ep[c]);
        v[1] = x4.y + ElemTraits<T>::to_f(ep[c + 1]);
        v[2] = x4.z + ElemTraits<T>::to_f(ep[c + 2]);
        v[3] = x4.w + ElemTraits<T>::to_f(ep[c + 3]);
        for (int k = 0; k < a.A; ++k) {
          const float ak = arow[k];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += ak * ElemTraits<T>::to_f(W[(size_t)(c + e) * a.A + k]);
        }
      }
      xv[i] = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = 4 * (t + 256 * i);
    if (c < d) {
      *reinterpret_cast<float4*>(a.x + (size_t)m * d + c) = xv[i];
      ss += xv[i].x * xv[i].x + xv[i].y * xv[i].y + xv[i].z * xv[i].z + xv[i].w * xv[i].w;
    }
  }
  ss = wave_sum(ss);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  const float rstd = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + a.eps);
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = 4 * (t + 256 * i);
    if (c >= d) continue;
    const float4 g = *reinterpret_cast<const float4*>(a.gamma + c);
    const float4 bb = *reinterpret_cast<const float4*>(a.beta + c);
    const float u0 = xv[i].x * rstd * (1.0f + g.x) + bb.x;
    const float u1 = xv[i].y * rstd * (1.0f + g.y) + bb.y;
    const float u2 = xv[i].z * rstd * (1.0f + g.z) + bb.z;
    const float u3 = xv[i].w * rstd * (1.0f + g.w) + bb.w;
    if (a.u_f32) {
      *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.u) + (size_t)m * d + c) = make_float4(u0, u1, u2, u3);
    } else {
      T* up = reinterpret_cast<T*>(a.u) + (size_t)m * d + c;
      up[0] = ElemTraits<T>::from_f(u0);
      up[1] = ElemTraits<T>::from_f(u1);
      up[2] = ElemTraits<T>::from_f(u2);
      up[3] = ElemTraits<T>::from_f(u3);
    }
    xv[i] = make_float4(u0, u1, u2, u3);  // keep u for the quantiser
  }
  if (a.q == nullptr) return;
  // Per-token absmax int8 quantisation of the fp32 u (same arithmetic as
  // quantize_kernel, so the codes are identical to quantising the stored u).
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = 4 * (t + 256 * i);
    if (c < d) amax = fmaxf(fmaxf(fmaxf(amax, fabsf(xv[i].x)), fmaxf(fabsf(xv[i].y), fabsf(xv[i].z))), fabsf(xv[i].w));
  }
  amax = wave_max(amax);
  __syncthreads();  // every thread has read red[] for rstd
  if ((t & 63) == 0) red[t >> 6] = amax;
  __syncthreads();
  const float r = fmaxf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])), 1e-5f);
  const float inv = __fdiv_rn(127.0f, r);
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = 4 * (t + 256 * i);
    if (c >= d) continue;
    const float e[4] = {xv[i].x, xv[i].y, xv[i].z, xv[i].w};
    uint32_t packed = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float qv = fminf(fmaxf(rintf(__fmul_rn(e[k], inv)), -128.0f), 127.0f);
      packed |= ((uint32_t)(int)qv & 0xFFu) << (8 * k);
    }
    *reinterpret_cast<uint32_t*>(a.q + (size_t)m * d + c) = packed;
  }
  if (t == 0) a.qr[m] = r;
}

__global__ void copy_f32_kernel(float* dst, const float* src, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// Rotary position embedding in place (rotate-half form): row r of x holds
// nheads heads of hd values from column col0 (row pitch ld); its position is
// pos0 + r % rpr.  With h = hd / 2 and w_i = base^(-2i/hd) the pair (i, i+h)
// turns by the angle pos * w_i (lbase = log2(base)).  One thread per pair.
template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(T* x, int rows, int rpr, int ld, int col0, int nheads, int hd,
                                                   int pos0, float lbase) {
  const int half = hd / 2;
  const long long total = (long long)rows * nheads * half;
  for (long long idx = blockIdx.x * 256LL + threadIdx.x; idx < total; idx += (long long)gridDim.x * 256LL) {
    const int i = (int)(idx % half);
    const long long rh = idx / half;
    const int h = (int)(rh % nheads);
    const int r = (int)(rh / nheads);
    const float pos = (float)(pos0 + r % rpr);
    const float w = exp2f(-2.0f * (float)i / (float)hd * lbase);
    float sn, cs;
    sincosf(pos * w, &sn, &cs);
    T* row = x + (size_t)r * ld + col0 + (size_t)h * hd;
    const float lo = ElemTraits<T>::to_f(row[i]), hi = ElemTraits<T>::to_f(row[i + half]);
    row[i] = ElemTraits<T>::from_f(lo * cs - hi * sn);
    row[i + half] = ElemTraits<T>::from_f(hi * cs + lo * sn);
  }
}

// y[i] = sum over the nsplit partial arrays part[s][i], in split order.
__global__ void sum_partials_kernel(float* y, const float* part, int nsplit, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    float v = 0.0f;
    for (int sp = 0; sp < nsplit; ++sp) v += part[(size_t)sp * n + i];
    y[i] = v;
  }
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
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float amax = 0.0f;
  for (int k = threadIdx.x; k < a.K; k += 256) {
    float v;
    if (a.src_type == 1)
      v = bf2f(reinterpret_cast<const bf16_t*>(a.x)[(size_t)m * a.ldx + k]);
    else
      v = reinterpret_cast<const float*>(a.x)[(size_t)m * a.ldx + k];
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

// The same quantiser for rows that fit in registers: each thread issues all
// of its 16-byte loads (VE values each) before the first use, so a row costs
// one load latency instead of one per loop trip.  Same arithmetic and codes.
constexpr int QUANT_NV = 8;   // 16-byte vectors per thread: K <= VE * 256 * QUANT_NV
template <int SRC>
__global__ __launch_bounds__(256) void quantize_vec_kernel(QuantArgs a) {
  constexpr int VE = SRC == 1 ? 8 : 4;            // values per 16-byte vector
  constexpr int ESZ = SRC == 1 ? 2 : 4;
  __shared__ float red[4];
  const int m = blockIdx.x, t = threadIdx.x;
  const char* row = reinterpret_cast<const char*>(a.x) + (size_t)m * a.ldx * ESZ;
  uint4 v[QUANT_NV];
#pragma unroll
  for (int i = 0; i < QUANT_NV; ++i) {
    const int c = VE * (t + 256 * i);
    v[i] = c < a.K ? *reinterpret_cast<const uint4*>(row + (size_t)c * ESZ) : make_uint4(0, 0, 0, 0);
  }
  float amax = 0.0f;
  float f[QUANT_NV][VE];
#pragma unroll
  for (int i = 0; i < QUANT_NV; ++i) {
    const uint32_t w[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      f[i][j] = SRC == 1 ? __uint_as_float(j & 1 ? (w[j >> 1] & 0xFFFF0000u) : (w[j >> 1] << 16))
                         : __uint_as_float(w[j & 3]);
      amax = fmaxf(amax, fabsf(f[i][j]));
    }
  }
  amax = wave_max(amax);
  if ((t & 63) == 0) red[t >> 6] = amax;
  __syncthreads();
  const float r = fmaxf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])), 1e-5f);
  const float inv = __fdiv_rn(127.0f, r);
#pragma unroll
  for (int i = 0; i < QUANT_NV; ++i) {
    const int c = VE * (t + 256 * i);
    if (c >= a.K) continue;
    uint32_t p[VE / 4];
#pragma unroll
    for (int j = 0; j < VE / 4; ++j) p[j] = 0;
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      const float qv = fminf(fmaxf(rintf(__fmul_rn(f[i][j], inv)), -128.0f), 127.0f);
      p[j >> 2] |= ((uint32_t)(int)qv & 0xFFu) << (8 * (j & 3));
    }
    int8_t* dst = a.q + (size_t)m * a.K + c;
    if (VE == 8)
      *reinterpret_cast<uint2*>(dst) = make_uint2(p[0], p[VE / 4 - 1]);
    else
      *reinterpret_cast<uint32_t*>(dst) = p[0];
  }
  if (t == 0) a.r[m] = r;
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

hipError_t launch_chunk_start(int et, const CallParams* cp, float* a, float* xs, const void* W_s,
                              const float* b_s, const float* b_in, int B, int n, int A, int S, int d, void* e,
                              int T, int Tpad, hipStream_t s) {
  const int XB = (d + XCOLS - 1) / XCOLS, EB = (d / 2 + 255) / 256;
  const int blocks = B * XB + (e ? Tpad * EB : 0);
  if (blocks <= 0) return hipSuccess;
  if (et == ET_BF16)
    hipLaunchKernelGGL(chunk_start_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, cp, a, xs,
                       reinterpret_cast<const bf16_t*>(W_s), b_s, b_in, B, n, A, S, d,
                       reinterpret_cast<bf16_t*>(e), T, Tpad);
  else
    hipLaunchKernelGGL(chunk_start_kernel<float>, dim3(blocks), dim3(256), 0, s, cp, a, xs,
                       reinterpret_cast<const float*>(W_s), b_s, b_in, B, n, A, S, d,
                       reinterpret_cast<float*>(e), T, Tpad);
  return hipGetLastError();
}

hipError_t launch_row_norm(int et, const RowNormArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.d > 4 * 256 * 4 || a.d % 4 || (a.mode == 1 && a.A > 64)) return hipErrorInvalidValue;
  if (et == ET_BF16)
    hipLaunchKernelGGL(row_norm_kernel<bf16_t>, dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(row_norm_kernel<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_time_embed(int et, const CallParams* cp, void* e, int T, int Tpad, int d, hipStream_t s) {
  return launch_chunk_start(et, cp, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0, 0, 0, d, e, T, Tpad, s);
}

hipError_t launch_copy_f32(float* dst, const float* src, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(copy_f32_kernel, dim3(blocks), dim3(256), 0, s, dst, src, n);
  return hipGetLastError();
}

hipError_t launch_rope(int et, void* x, int rows, int rpr, int ld, int col0, int nheads, int hd, int pos0, float base,
                       hipStream_t s) {
  if (rows <= 0 || nheads <= 0) return hipSuccess;
  if (hd % 2 || base <= 1.0f || rpr < 1) return hipErrorInvalidValue;
  const long long total = (long long)rows * nheads * (hd / 2);
  const int blocks = (int)((total + 255) / 256 > 2048 ? 2048 : (total + 255) / 256);
  const float lbase = std::log2(base);
  if (et == ET_BF16)
    hipLaunchKernelGGL(rope_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, reinterpret_cast<bf16_t*>(x), rows, rpr,
                       ld, col0, nheads, hd, pos0, lbase);
  else
    hipLaunchKernelGGL(rope_kernel<float>, dim3(blocks), dim3(256), 0, s, reinterpret_cast<float*>(x), rows, rpr, ld,
                       col0, nheads, hd, pos0, lbase);
  return hipGetLastError();
}

hipError_t launch_sum_partials(float* y, const float* part, int nsplit, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(sum_partials_kernel, dim3(blocks), dim3(256), 0, s, y, part, nsplit, n);
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
  // register-resident rows: whole 16-byte vectors, aligned rows and codes
  const int ve = a.src_type == 1 ? 8 : 4;
  const bool vec = a.K % ve == 0 && a.ldx % ve == 0 && a.K <= ve * 256 * QUANT_NV &&
                   reinterpret_cast<uintptr_t>(a.x) % 16 == 0 && reinterpret_cast<uintptr_t>(a.q) % ve == 0;
  if (vec && a.src_type == 1)
    hipLaunchKernelGGL(quantize_vec_kernel<1>, dim3(a.M), dim3(256), 0, s, a);
  else if (vec)
    hipLaunchKernelGGL(quantize_vec_kernel<0>, dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(quantize_kernel, dim3(a.M), dim3(256), (size_t)a.K * sizeof(float), s, a);
  return hipGetLastError();
}

hipError_t launch_check_finite(const float* x, size_t n, int* flag, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256);
  hipLaunchKernelGGL(check_finite_kernel, dim3(blocks), dim3(256), 0, s, x, n, flag);
  return hipGetLastError();
}

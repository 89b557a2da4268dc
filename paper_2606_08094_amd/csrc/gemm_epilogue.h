// Fused epilogues of the expert's projections, shared by the dense MFMA GEMM
// and the ternary W2A8 GEMM.  The caller passes the reduced fp32 tile of one
// workgroup: lane holds rows 4*(lane/16)+i of each 16-row subtile ms and
// column lane%16 of W-row subtile s, for W rows nw0 + 16*s + lane%16.
#pragma once
#include "device_common.h"

template <typename T, int MS, int NSUB>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, f32x4 (&acc)[MS][NSUB], int m0, int ntile,
                                              int nw0, float* red_s) {
  constexpr int MT = 16 * MS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N;
  switch (a.epi) {
    case EPI_STORE: {
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
          for (int s = 0; s < NSUB; ++s) {
            const int n = nw0 + s * 16 + r16;
            if (m < M && n < N) {
              float v = acc[ms][s][i] + (a.bias ? a.bias[n] : 0.0f);
              v = act_f(a.act, v);
              if (a.out_f32)
                reinterpret_cast<float*>(a.out)[(size_t)m * a.ldo + n] = v;
              else
                reinterpret_cast<T*>(a.out)[(size_t)m * a.ldo + n] = ElemTraits<T>::from_f(v);
            }
          }
        }
      break;
    }
    case EPI_KVCACHE: {
      const int G = a.d_kv / a.hd;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
          for (int s = 0; s < NSUB; ++s) {
            const int n = nw0 + s * 16 + r16;
            if (m < M && n < N) {
              const int b = m / a.P, p = m - b * a.P;
              const int kv = n / a.d_kv, rem = n - kv * a.d_kv;
              const int g = rem / a.hd, c = rem - g * a.hd;
              const size_t idx = ((((size_t)kv * a.B + b) * G + g) * a.P + p) * a.hd + c;
              reinterpret_cast<T*>(a.cache)[idx] = ElemTraits<T>::from_f(acc[ms][s][i]);
            }
          }
        }
      break;
    }
    case EPI_GLU: {
      const int F = N / 2;
      const int f = ntile * 64 + wave * 16 + r16;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
          if (m < M && f < F) {
            const float h = act_f(a.act, acc[ms][0][i]) * acc[ms][NSUB - 1][i];
            if (a.out_f32)
              reinterpret_cast<float*>(a.out)[(size_t)m * a.ldo + f] = h;
            else
              reinterpret_cast<T*>(a.out)[(size_t)m * a.ldo + f] = ElemTraits<T>::from_f(h);
          }
        }
      break;
    }
    case EPI_RESID: {
      const int n = nw0 + r16;  // NSUB == 1
      const float al = (n < N) ? a.alpha[n] : 0.0f;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = ms * 16 + g4 * 4 + i;
          const int m = m0 + row;
          float sq = 0.0f;
          if (m < M && n < N) {
            float* xp = a.xres + (size_t)m * a.ldxr + n;
            const float xv = *xp + al * acc[ms][0][i];
            *xp = xv;
            sq = xv * xv;
          }
          sq = sum16(sq);
          if (r16 == 0) red_s[wave * MT + row] = sq;
        }
      __syncthreads();
      if (tid < MT && m0 + tid < M) {
        const float t = red_s[tid] + red_s[MT + tid] + red_s[2 * MT + tid] + red_s[3 * MT + tid];
        a.rowss_out[(size_t)ntile * M + m0 + tid] = t;
      }
      break;
    }
    case EPI_EULER: {
      const CallParams* cp = a.cp;
      const float dt = cp->tau[a.step + 1] - cp->tau[a.step];
      const int n = nw0 + r16;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
          if (m < M && n < N) {
            const float v = acc[ms][0][i] + a.bias[n];
            float* ap = a.a + (size_t)m * N + n;
            const float an = a.regression ? v : (*ap + dt * v);
            *ap = an;
            if (a.last) {
              float o = an;
              if (cp->act_std) o *= cp->act_std[n];
              if (cp->act_mean) o += cp->act_mean[n];
              cp->actions_out[(size_t)m * N + n] = o;
            }
          }
        }
      break;
    }
    default:
      break;
  }
}

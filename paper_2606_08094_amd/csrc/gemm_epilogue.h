// Fused epilogues of the expert's projections, shared by the dense MFMA GEMMs
// and the ternary W2A8 GEMM.  One call handles the reduced fp32 tile of one
// wave: lane holds rows 4*(lane/16)+i of each 16-row subtile ms (rows from m0)
// and column lane%16 of each of the NSUB W-row subtiles starting at W row nb.
// EPI_PARTIAL writes the raw fp32 tile of K-split `split` to
// out + split * M * ldo (a later launch sums the splits).
#pragma once
#include "device_common.h"

template <typename T, int MS, int NSUB>
__device__ __forceinline__ void wave_epilogue(const GemmArgs& a, const f32x4 (&acc)[MS][NSUB], int m0, int nb,
                                              int split) {
  const int lane = threadIdx.x & 63;
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
            const int n = nb + s * 16 + r16;
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
            const int n = nb + s * 16 + r16;
            if (m < M && n < N) {
              const int b = m / a.P, p = m - b * a.P;
              const int slot = a.lay_cols > 0 ? n / a.lay_cols : 0;
              const int nl = n - slot * a.lay_cols;
              const int kv = nl / a.d_kv, rem = nl - kv * a.d_kv;
              const int g = rem / a.hd, c = rem - g * a.hd;
              const size_t idx = (size_t)slot * a.lay_stride + ((((size_t)kv * a.B + b) * G + g) * a.P + p) * a.hd + c;
              reinterpret_cast<T*>(a.cache)[idx] = ElemTraits<T>::from_f(acc[ms][s][i]);
            }
          }
        }
      break;
    }
    case EPI_GLU: {
      // W rows are interleaved 16-row blocks: gate block j at nb + 32 j, its
      // up block at nb + 32 j + 16 (subtiles 2 j and 2 j + 1; NSUB = 2 or 4).
      const int F = N / 2;
#pragma unroll
      for (int j = 0; j < NSUB / 2; ++j) {   // no pairs (and no output) in NSUB = 1 tiles
        const int f = (nb / 32 + j) * 16 + r16;
#pragma unroll
        for (int ms = 0; ms < MS; ++ms)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = m0 + ms * 16 + g4 * 4 + i;
            if (m < M && f < F) {
              const float h = act_f(a.act, acc[ms][2 * j][i]) * acc[ms][2 * j + 1][i];
              if (a.out_f32)
                reinterpret_cast<float*>(a.out)[(size_t)m * a.ldo + f] = h;
              else
                reinterpret_cast<T*>(a.out)[(size_t)m * a.ldo + f] = ElemTraits<T>::from_f(h);
            }
          }
      }
      break;
    }
    case EPI_PARTIAL: {
      float* out = reinterpret_cast<float*>(a.out) + (size_t)split * M * a.ldo;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
          for (int s = 0; s < NSUB; ++s) {
            const int n = nb + s * 16 + r16;
            if (m < M && n < N) out[(size_t)m * a.ldo + n] = acc[ms][s][i];
          }
        }
      break;
    }
    case EPI_RESID: {
      const int n = nb + r16;  // NSUB == 1
      const float al = (n < N) ? a.alpha[n] : 0.0f;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
          if (m < M && n < N) {
            float* xp = a.xres + (size_t)m * a.ldxr + n;
            *xp = *xp + al * acc[ms][0][i];
          }
        }
      break;
    }
    case EPI_EULER: {
      const CallParams* cp = a.cp;
      const float dt = cp->tau[a.step + 1] - cp->tau[a.step];
      const int n = nb + r16;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + ms * 16 + g4 * 4 + i;
          // state-token rows carry no action: skipped, the rest map to action rows
          const int t = a.stok ? m % a.stok : 1;
          const int am = a.stok ? (m / a.stok) * (a.stok - 1) + t - 1 : m;
          if (m < M && n < N && t != 0) {
            const float v = acc[ms][0][i] + a.bias[n];
            float* ap = a.a + (size_t)am * N + n;
            const float an = a.regression ? v : (*ap + dt * v);
            *ap = an;
            if (a.last) {
              float o = an;
              if (cp->act_std) o *= cp->act_std[n];
              if (cp->act_mean) o += cp->act_mean[n];
              cp->actions_out[(size_t)am * N + n] = o;
            }
          }
        }
      break;
    }
    default:
      break;
  }
}

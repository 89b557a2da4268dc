// Attention of the action tokens over [cached prefix K/V ; action-token K/V].
//
// Self (keys = the chunk's own tokens), cross (keys = the cached prefix rows)
// and joint (one softmax over both) share one kernel.  Head h reads K/V head
// floor(h*G/H).  No mask: every key is visible to every query.
//
// One wave handles (request b, head h, a tile of 16 queries, one key split).
// Scores are computed transposed, S^T = K Q^T on MFMA, so that each lane's
// column is one query: the running max and sum of the online softmax live in
// the lane, and P^T comes out of the accumulator already in the B-operand
// layout of O^T += V^T P^T.  V blocks of 32 keys are staged in LDS.  Key splits
// write unnormalised partials plus (max, sum); the last wave to arrive merges
// them in split order.
#include "device_common.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;

template <typename T, int HD>
__global__ __launch_bounds__(64) void attn_kernel(AttnArgs a) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int NQV = HD / (4 * E);   // 16-byte vectors per lane along hd
  constexpr int DT = HD / 16;         // 16-wide dim tiles of O^T
  __shared__ __align__(16) T vlds[32 * HD];
  __shared__ int flag_s;

  const int lane = threadIdx.x, r16 = lane & 15, g4 = lane >> 4;
  const int QT = (a.n + 15) / 16;
  int u = blockIdx.x;
  const int split = u % a.kv_split;
  u /= a.kv_split;
  const int qt = u % QT;
  u /= QT;
  const int h = u % a.H;
  const int b = u / a.H;
  const int g = (h * a.G) / a.H;

  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int total = npre + nself;
  const int kbeg = split * a.key_chunk;
  const int kend = min(total, kbeg + a.key_chunk);

  const T* kc = reinterpret_cast<const T*>(a.kc);
  const T* vc = reinterpret_cast<const T*>(a.vc);
  if (npre > 0 && kc == nullptr) {
    kc = reinterpret_cast<const T*>(a.cp->kv_cache) + a.layer_off;
    vc = kc + (size_t)a.B * a.G * a.P * HD;
  }
  const T* ksf = reinterpret_cast<const T*>(a.ks);
  const T* vsf = reinterpret_cast<const T*>(a.vs);
  auto key_row = [&](const T* cache, const T* selfp, int key) -> const T* {
    if (key < npre) return cache + (((size_t)b * a.G + g) * a.P + key) * HD;
    return selfp + (size_t)(b * a.n + key - npre) * a.ldkv + g * HD;
  };

  // Q fragments (B operand of S^T): lane holds query row r16, dims g4*HD/4 + c*E ...
  const int qrow = qt * 16 + r16;
  const T* qp = reinterpret_cast<const T*>(a.q) + (size_t)(b * a.n + qrow) * a.ldq + h * HD + g4 * (HD / 4);
  uint4 qf[NQV];
#pragma unroll
  for (int c = 0; c < NQV; ++c) qf[c] = (qrow < a.n) ? ldg16(qp + c * E) : make_uint4(0, 0, 0, 0);

  f32x4 o[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.0f;
  const float sc = a.scale * kLog2e;

  for (int kb = kbeg; kb < kend; kb += 32) {
    // Scores of 32 keys: two 16-key tiles, lane holds keys 16t + 4*g4 + i for query r16.
    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int key = kb + t * 16 + r16;
      const bool kv_ok = key < kend;
      const T* kp = kv_ok ? key_row(kc, ksf, key) + g4 * (HD / 4) : nullptr;
#pragma unroll
      for (int c = 0; c < NQV; ++c) {
        const uint4 kf = kv_ok ? ldg16(kp + c * E) : make_uint4(0, 0, 0, 0);
        mma16(s[t], kf, qf[c], T());
      }
    }
    // Stage V rows kb .. kb+31 in LDS (zeros past the end).
    __syncthreads();
    for (int i = lane; i < 32 * (HD / E); i += 64) {
      const int kr = i / (HD / E), cv = i - kr * (HD / E);
      const int key = kb + kr;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (key < kend) val = ldg16(key_row(vc, vsf, key) + cv * E);
      *reinterpret_cast<uint4*>(vlds + kr * HD + cv * E) = val;
    }
    // Online softmax update for query r16.
    float bmax = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb + t * 16 + g4 * 4 + i;
        const float v = (key < kend) ? s[t][i] * sc : -INFINITY;
        s[t][i] = v;
        bmax = fmaxf(bmax, v);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float mnew = fmaxf(mrun, bmax);
    const float corr = exp2f(mrun - mnew);
    float psum = 0.0f;
    float p[8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = exp2f(s[t][i] - mnew);
        p[t * 4 + i] = pv;
        psum += pv;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    lrun = lrun * corr + psum;
    mrun = mnew;
#pragma unroll
    for (int d = 0; d < DT; ++d) o[d] *= corr;
    __syncthreads();
    // O^T += V^T P^T over these 32 keys.  k-slot j of lane group g4 is key
    // 4*g4 + j (j < 4) or 16 + 4*g4 + (j - 4).
    if constexpr (E == 8) {
      uint4 pb;
      pb.x = pack_bf16x2(p[0], p[1]);
      pb.y = pack_bf16x2(p[2], p[3]);
      pb.z = pack_bf16x2(p[4], p[5]);
      pb.w = pack_bf16x2(p[6], p[7]);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const int dim = d * 16 + r16;
        const bf16_t* vb = reinterpret_cast<const bf16_t*>(vlds) + dim;
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int k0 = (j < 2) ? (4 * g4 + 2 * j) : (16 + 4 * g4 + 2 * (j - 2));
          w[j] = (uint32_t)vb[k0 * HD] | ((uint32_t)vb[(k0 + 1) * HD] << 16);
        }
        mma16(o[d], make_uint4(w[0], w[1], w[2], w[3]), pb, T());
      }
    } else {
      const float* vf = reinterpret_cast<const float*>(vlds);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const int dim = d * 16 + r16;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf[(t * 16 + 4 * g4 + i) * HD + dim], p[t * 4 + i],
                                                        o[d], 0, 0, 0);
      }
    }
  }

  // Lane holds O^T[dim = 16d + 4*g4 + i][query r16].
  auto store = [&](const f32x4* ov, float inv) {
    if (qrow >= a.n) return;
    T* op = reinterpret_cast<T*>(a.o) + (size_t)(b * a.n + qrow) * a.ldo + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) op[d * 16 + 4 * g4 + i] = ElemTraits<T>::from_f(ov[d][i] * inv);
  };

  if (a.kv_split == 1) {
    store(o, 1.0f / lrun);
    return;
  }
  const int tile = (b * a.H + h) * QT + qt;
  constexpr int PER = DT * 64 * 4 + 2 * 64;  // floats per (tile, split)
  float* wsp = a.ws + (size_t)tile * a.kv_split * PER;
  {
    float* mine = wsp + (size_t)split * PER;
    f32x4* ov = reinterpret_cast<f32x4*>(mine);
#pragma unroll
    for (int d = 0; d < DT; ++d) ov[d * 64 + lane] = o[d];
    mine[DT * 256 + lane] = mrun;
    mine[DT * 256 + 64 + lane] = lrun;
  }
  if (!splitk_arrive_last(&a.cnt[tile], (unsigned)a.kv_split, &flag_s)) return;
  float mmax = -INFINITY;
  for (int sp = 0; sp < a.kv_split; ++sp) mmax = fmaxf(mmax, wsp[(size_t)sp * PER + DT * 256 + lane]);
  float lsum = 0.0f;
  f32x4 acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int sp = 0; sp < a.kv_split; ++sp) {
    const float* part = wsp + (size_t)sp * PER;
    const float f = exp2f(part[DT * 256 + lane] - mmax);
    lsum += f * part[DT * 256 + 64 + lane];
    const f32x4* ov = reinterpret_cast<const f32x4*>(part);
#pragma unroll
    for (int d = 0; d < DT; ++d) acc[d] += f * ov[d * 64 + lane];
  }
  store(acc, 1.0f / lsum);
}

template <typename T, int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  const int QT = (a.n + 15) / 16;
  const int units = a.B * a.H * QT * a.kv_split;
  if (units <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_kernel<T, HD>), dim3(units), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

size_t attention_ws_floats(const AttnArgs& a) {
  const int QT = (a.n + 15) / 16;
  const size_t per = (size_t)(a.hd / 16) * 64 * 4 + 2 * 64;
  return a.kv_split > 1 ? (size_t)a.B * a.H * QT * a.kv_split * per : 0;
}

hipError_t launch_attention(int et, const AttnArgs& a, hipStream_t s) {
  if (et == ET_BF16) {
    switch (a.hd) {
      case 64: return launch_hd<bf16_t, 64>(a, s);
      case 128: return launch_hd<bf16_t, 128>(a, s);
      case 256: return launch_hd<bf16_t, 256>(a, s);
    }
  } else {
    switch (a.hd) {
      case 64: return launch_hd<float, 64>(a, s);
      case 128: return launch_hd<float, 128>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

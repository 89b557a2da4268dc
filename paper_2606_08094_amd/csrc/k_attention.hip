// Attention of the action tokens over [cached prefix K/V ; action-token K/V].
//
// Self (keys = the chunk's own tokens), cross (keys = the cached prefix rows)
// and joint (one softmax over both) share one kernel.  Query head h reads K/V
// head floor(h*G/H).  No mask: every key is visible to every query.
//
// One workgroup handles (request b, 16-query tile, K/V head g, key split) with
// one wave per query head of the group, so a K/V block of 32 keys is staged in
// LDS once and serves every head that shares it.  Blocks are double-buffered:
// the loads of block j+1 are in flight while block j is multiplied.  Prefix
// blocks and action-token blocks never mix, so a block has a single source.
//
// Scores are computed transposed, S^T = K Q^T on MFMA, so each lane's column is
// one query and the online-softmax statistics live in the lane.  Row rho of
// score tile t holds key 8*(rho/4) + 4*t + rho%4 of the block; lane group q
// (= lane/16) then holds keys 8q .. 8q+7 across the two tiles, exactly the k
// slots of its B operand in O^T += V^T P^T, and V is stored transposed in LDS
// ([dim][key]) so the A operand is one 16-byte read.
//
// With more than one key split each split writes its output normalised by its
// own sum (bf16) plus its (max, sum); attn_merge combines them.
#include "device_common.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;

template <typename T, int HD>
struct AttnLds {
  static constexpr int E = ElemTraits<T>::E;
  static constexpr int KP = HD + E;       // K row pitch (elements)
  static constexpr int VP = 32 + E;       // V^T row pitch (elements)
  static constexpr size_t KBYTES = 32 * KP * sizeof(T);
  static constexpr size_t VBYTES = HD * VP * sizeof(T);
  static constexpr size_t BUF = KBYTES + VBYTES;
};

template <typename T, int HD>
__global__ __launch_bounds__(512) void attn_kernel(AttnArgs a) {
  using L = AttnLds<T, HD>;
  constexpr int E = L::E;
  constexpr int NQV = HD / (4 * E);   // 16-byte vectors per lane along hd
  constexpr int DT = HD / 16;         // 16-wide dim tiles of O^T
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nthr = blockDim.x;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int per = a.H / a.G;          // query heads per K/V head (= waves)
  const int QT = (a.n + 15) / 16;
  int u = blockIdx.x;
  const int split = u % a.kv_split;
  u /= a.kv_split;
  const int g = u % a.G;
  u /= a.G;
  const int qt = u % QT;
  const int b = u / QT;
  const int h = g * per + wave;

  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nbp = (npre + 31) / 32, nbs = (nself + 31) / 32;
  const int jbeg = split * a.key_chunk, jend = min(nbp + nbs, jbeg + a.key_chunk);

  const T* kc = reinterpret_cast<const T*>(a.kc);
  const T* vc = reinterpret_cast<const T*>(a.vc);
  if (npre > 0 && kc == nullptr) {
    kc = reinterpret_cast<const T*>(a.cp->kv_cache) + a.layer_off;
    vc = kc + (size_t)a.B * a.G * a.P * HD;
  }
  kc += ((size_t)b * a.G + g) * a.P * HD;
  vc += ((size_t)b * a.G + g) * a.P * HD;
  const T* ksf = reinterpret_cast<const T*>(a.ks) + (size_t)b * a.n * a.ldkv + g * HD;
  const T* vsf = reinterpret_cast<const T*>(a.vs) + (size_t)b * a.n * a.ldkv + g * HD;

  // Staging of one K/V block: every thread owns items tid, tid + nthr, ...
  // (16-byte vectors of a K row and of a V row).  The first SU items are
  // loaded into registers by `fetch` (issued before the math on the previous
  // block) and written to LDS by `store`; any further items are copied
  // synchronously by `store`.
  constexpr int ITEMS = 32 * (HD / E);
  constexpr int SU = 4;
  uint4 kreg[SU], vreg[SU];
  auto src = [&](int j, int kr, const T*& kp, const T*& vp) -> bool {
    const bool pre = j < nbp;
    const int key0 = pre ? j * 32 : (j - nbp) * 32;
    const int cnt = pre ? min(32, npre - key0) : min(32, nself - key0);
    if (kr >= cnt) return false;
    const int key = key0 + kr;
    kp = pre ? kc + (size_t)key * HD : ksf + (size_t)key * a.ldkv;
    vp = pre ? vc + (size_t)key * HD : vsf + (size_t)key * a.ldkv;
    return true;
  };
  auto block_cnt = [&](int j) {
    const bool pre = j < nbp;
    const int key0 = pre ? j * 32 : (j - nbp) * 32;
    return pre ? min(32, npre - key0) : min(32, nself - key0);
  };
  auto fetch = [&](int j) {
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * nthr;
      const int kr = i / (HD / E), cv = i - kr * (HD / E);
      const T *kp, *vp;
      if (i < ITEMS && src(j, kr, kp, vp)) {
        kreg[u] = ldg16(kp + cv * E);
        vreg[u] = ldg16(vp + cv * E);
      } else {
        kreg[u] = make_uint4(0, 0, 0, 0);
        vreg[u] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto put = [&](int buf, int i, uint4 kv4, uint4 vv4) {
    T* kl = reinterpret_cast<T*>(smem + buf * L::BUF);
    T* vl = reinterpret_cast<T*>(smem + buf * L::BUF + L::KBYTES);
    const int kr = i / (HD / E), cv = i - kr * (HD / E);
    *reinterpret_cast<uint4*>(kl + kr * L::KP + cv * E) = kv4;
    const uint32_t w4[4] = {vv4.x, vv4.y, vv4.z, vv4.w};
    if constexpr (E == 8) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        reinterpret_cast<bf16_t*>(vl)[(cv * 8 + e) * L::VP + kr] = (bf16_t)(w4[e >> 1] >> (16 * (e & 1)));
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) reinterpret_cast<float*>(vl)[(cv * 4 + e) * L::VP + kr] = __uint_as_float(w4[e]);
    }
  };
  auto store = [&](int j, int buf) {
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * nthr;
      if (i < ITEMS) put(buf, i, kreg[u], vreg[u]);
    }
    for (int i = threadIdx.x + SU * nthr; i < ITEMS; i += nthr) {
      const int kr = i / (HD / E), cv = i - kr * (HD / E);
      const T *kp, *vp;
      uint4 kv4 = make_uint4(0, 0, 0, 0), vv4 = make_uint4(0, 0, 0, 0);
      if (src(j, kr, kp, vp)) {
        kv4 = ldg16(kp + cv * E);
        vv4 = ldg16(vp + cv * E);
      }
      put(buf, i, kv4, vv4);
    }
  };

  // Q fragments (B operand of S^T): query row r16 of head h, dims g4*HD/4 + c*E ..
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

  if (jbeg < jend) {
    fetch(jbeg);
    store(jbeg, 0);
  }
  for (int j = jbeg; j < jend; ++j) {
    const int buf = (j - jbeg) & 1;
    const int cnt = block_cnt(j);
    __syncthreads();                   // block j staged; block j-1 fully read
    if (j + 1 < jend) fetch(j + 1);    // global loads in flight during the math below
    const T* kl = reinterpret_cast<const T*>(smem + buf * L::BUF);
    const T* vl = reinterpret_cast<const T*>(smem + buf * L::BUF + L::KBYTES);

    // scores: tile t, row rho = r16 -> key 8*(rho/4) + 4t + rho%4
    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int kr = 8 * (r16 >> 2) + 4 * t + (r16 & 3);
      const T* krow = kl + kr * L::KP + g4 * (HD / 4);
#pragma unroll
      for (int c = 0; c < NQV; ++c) mma16(s[t], *reinterpret_cast<const uint4*>(krow + c * E), qf[c], T());
    }
    // lane holds keys 8*g4 + 4t + i for query r16
    float bmax = -INFINITY;
    float p[8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kr = 8 * g4 + 4 * t + i;
        const float v = (kr < cnt) ? s[t][i] * sc : -INFINITY;
        p[4 * t + i] = v;
        bmax = fmaxf(bmax, v);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float mnew = fmaxf(mrun, bmax);
    const float corr = exp2f(mrun - mnew);
    float psum = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      p[k] = exp2f(p[k] - mnew);
      psum += p[k];
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    lrun = lrun * corr + psum;
    mrun = mnew;
#pragma unroll
    for (int d = 0; d < DT; ++d) o[d] *= corr;
    // O^T += V^T P^T: k slot k of lane group g4 is key 8*g4 + k.
    if constexpr (E == 8) {
      uint4 pb;
      pb.x = pack_bf16x2(p[0], p[1]);
      pb.y = pack_bf16x2(p[2], p[3]);
      pb.z = pack_bf16x2(p[4], p[5]);
      pb.w = pack_bf16x2(p[6], p[7]);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const uint4 va = *reinterpret_cast<const uint4*>(vl + (d * 16 + r16) * L::VP + 8 * g4);
        mma16(o[d], va, pb, T());
      }
    } else {
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const float* vrow = reinterpret_cast<const float*>(vl) + (d * 16 + r16) * L::VP + 8 * g4;
#pragma unroll
        for (int k = 0; k < 8; ++k) o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vrow[k], p[k], o[d], 0, 0, 0);
      }
    }
    if (j + 1 < jend) store(j + 1, buf ^ 1);
  }

  // Lane holds O^T[dim = 16d + 4*g4 + i][query r16].
  if (qrow >= a.n) return;
  const float inv = lrun > 0.0f ? 1.0f / lrun : 0.0f;
  if (a.kv_split == 1) {
    T* op = reinterpret_cast<T*>(a.o) + (size_t)(b * a.n + qrow) * a.ldo + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) op[d * 16 + 4 * g4 + i] = ElemTraits<T>::from_f(o[d][i] * inv);
    return;
  }
  // partial: normalised by its own sum, plus (max, sum)
  const int rows = a.B * a.n, dq = a.H * HD;
  T* pp = reinterpret_cast<T*>(a.part) + ((size_t)split * rows + b * a.n + qrow) * dq + h * HD;
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 4; ++i) pp[d * 16 + 4 * g4 + i] = ElemTraits<T>::from_f(o[d][i] * inv);
  if (g4 == 0) {
    float* st = a.stats + (((size_t)split * rows + b * a.n + qrow) * a.H + h) * 2;
    st[0] = mrun;
    st[1] = lrun;
  }
}

// O[m][h] = sum_s w_s O_s / sum_s w_s with w_s = l_s * 2^(m_s - max_s m_s).
// One thread per 16-byte vector of the output row; the splits' vectors are
// loaded four at a time.
template <typename T>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int E = ElemTraits<T>::E;
  const int m = blockIdx.x;
  const int rows = a.B * a.n, dq = a.H * a.hd;
  __shared__ float wgt[64 * 32];   // kv_split <= 64, H <= 32
  for (int h = threadIdx.x; h < a.H; h += blockDim.x) {
    float mx = -INFINITY;
    for (int s = 0; s < a.kv_split; ++s) mx = fmaxf(mx, a.stats[(((size_t)s * rows + m) * a.H + h) * 2]);
    float tot = 0.0f;
    for (int s = 0; s < a.kv_split; ++s) {
      const float* st = a.stats + (((size_t)s * rows + m) * a.H + h) * 2;
      const float w = st[1] * exp2f(st[0] - mx);
      wgt[s * a.H + h] = w;
      tot += w;
    }
    for (int s = 0; s < a.kv_split; ++s) wgt[s * a.H + h] /= tot;
  }
  __syncthreads();
  const T* part = reinterpret_cast<const T*>(a.part);
  T* op = reinterpret_cast<T*>(a.o) + (size_t)m * a.ldo;
  for (int c = threadIdx.x * E; c < dq; c += blockDim.x * E) {
    const int h = c / a.hd;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    int s = 0;
    for (; s + 4 <= a.kv_split; s += 4) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = ldg16(part + ((size_t)(s + u) * rows + m) * dq + c);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float f[E];
        unpack16(v[u], f, T());
        const float w = wgt[(s + u) * a.H + h];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] += w * f[e];
      }
    }
    for (; s < a.kv_split; ++s) {
      float f[E];
      unpack16(ldg16(part + ((size_t)s * rows + m) * dq + c), f, T());
      const float w = wgt[s * a.H + h];
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += w * f[e];
    }
    stg16(op + c, pack16(acc, T()));
  }
}

template <typename T, int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s, int which) {
  const int QT = (a.n + 15) / 16;
  const int units = a.B * QT * a.G * a.kv_split;
  if (units <= 0) return hipSuccess;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, HD>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int threads = 64 * (a.H / a.G);
  using L = AttnLds<T, HD>;
  const size_t lds = 2 * L::BUF;
  if (which != 2) {
    hipLaunchKernelGGL((attn_kernel<T, HD>), dim3(units), dim3(threads), lds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (which == 1 || a.kv_split == 1) return hipSuccess;
  hipLaunchKernelGGL(attn_merge_kernel<T>, dim3(a.B * a.n), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// Keys per split in 32-key blocks, the number of splits, and the workspace.
void attention_split(AttnArgs& a, int want_splits) {
  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nblocks = (npre + 31) / 32 + (nself + 31) / 32;
  const int QT = (a.n + 15) / 16;
  int s = want_splits;
  if (s <= 0) {
    const int base = a.B * QT * a.G;
    s = (96 + base - 1) / base;   // about 96 workgroups
  }
  s = s < 1 ? 1 : (s > nblocks ? nblocks : s);
  s = s > 64 ? 64 : s;
  a.key_chunk = (nblocks + s - 1) / s;
  a.kv_split = (nblocks + a.key_chunk - 1) / a.key_chunk;
}

size_t attention_part_bytes(int et, const AttnArgs& a) {
  if (a.kv_split <= 1) return 0;
  return (size_t)a.kv_split * a.B * a.n * a.H * a.hd * (et == ET_BF16 ? 2 : 4);
}

size_t attention_stats_bytes(const AttnArgs& a) {
  if (a.kv_split <= 1) return 0;
  return (size_t)a.kv_split * a.B * a.n * a.H * 2 * sizeof(float);
}

hipError_t launch_attention(int et, const AttnArgs& a, hipStream_t s, int which) {
  if (a.H % a.G != 0 || a.H / a.G > 8 || a.H > 32 || a.kv_split > 64) return hipErrorInvalidValue;
  if (et == ET_BF16) {
    switch (a.hd) {
      case 64: return launch_hd<bf16_t, 64>(a, s, which);
      case 128: return launch_hd<bf16_t, 128>(a, s, which);
      case 256: return launch_hd<bf16_t, 256>(a, s, which);
    }
  } else {
    switch (a.hd) {
      case 64: return launch_hd<float, 64>(a, s, which);
      case 128: return launch_hd<float, 128>(a, s, which);
    }
  }
  return hipErrorInvalidValue;
}

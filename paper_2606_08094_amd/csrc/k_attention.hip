// Attention of the action tokens over [cached prefix K/V ; action-token K/V].
//
// Self (keys = the chunk's own tokens), cross (keys = the cached prefix rows)
// and joint (one softmax over both) share one kernel.  Query head h reads K/V
// head floor(h*G/H).  No mask: every key is visible to every query.
//
// One workgroup handles (request b, 16-query tile, K/V head g, key split) with
// one wave per query head of the group, so the split's K/V blocks (32 keys
// each) are staged in LDS once and serve every head that shares them.  A split
// of any length is processed in chunks of up to KB_MAX blocks: all global
// loads of a chunk are issued before its first LDS store, and the online
// softmax state carries from chunk to chunk.  Workgroups that read the same
// K/V (same request, head and split) get consecutive unit numbers, and the
// unit numbering follows the dispatcher's round robin over the 8 XCDs so that
// those workgroups share one XCD's L2.  Prefix blocks and action-token blocks
// never mix, so a block has a single source.
//
// Scores are computed transposed, S^T = K Q^T on MFMA, so each lane's column is
// one query and the online-softmax statistics live in the lane.  Row rho of
// score tile t holds key 8*(rho/4) + 4*t + rho%4 of the block; lane group q
// (= lane/16) then holds keys 8q .. 8q+7 across the two tiles, exactly the k
// slots of its B operand in O^T += V^T P^T.  bf16 V is staged row-major and
// read as V^T with two transposing LDS loads per operand (layout as in
// attn_tile); fp32 V is stored transposed ([dim][key], written as key pairs)
// so the A operand is one 16-byte read.
//
// With more than one key split each split writes its output normalised by its
// own sum (element type) plus its (max, sum); attn_merge combines them.
#include "device_common.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// K slot swizzle of attn_tile: K rows are stored unpadded with 16-byte chunk
// c of key k at slot c ^ kswz(k).  A score-operand read takes, in one bank
// cycle (eight lanes of 16 bytes), keys 8 (r / 4) + r % 4 for r = 0 .. 7 at
// one chunk, and kswz maps those eight keys to eight different slots.
VLA_DEV int kswz(int k) { return (k & 3) | ((k >> 1) & 4); }

template <typename T, int HD>
struct AttnLds {
  static constexpr int E = ElemTraits<T>::E;
  static constexpr int KP = HD + E;       // K row pitch (elements)
  static constexpr int VP = 32 + E;       // fp32: V^T row pitch (elements)
  static constexpr size_t KBYTES = 32 * KP * sizeof(T);
  // bf16: V row-major [32 keys][HD], 16-byte chunk c of key k at slot
  // c ^ 2 (k % 4), read with transposing loads; fp32: V^T [HD][VP]
  static constexpr size_t VBYTES = E == 8 ? (size_t)32 * HD * sizeof(T) : (size_t)HD * VP * sizeof(T);
  static constexpr size_t BUF = KBYTES + VBYTES;  // one 32-key block
};

// Most 32-key blocks one workgroup stages in LDS (KB_MAX * BUF <= 160 KB for
// every supported element type and head_dim).
constexpr int KB_MAX = 4;
static_assert(KB_MAX * AttnLds<bf16_t, 256>::BUF <= 160 * 1024, "LDS");
static_assert(KB_MAX * AttnLds<float, 128>::BUF <= 160 * 1024, "LDS");

template <typename T, int HD>
__global__ __launch_bounds__(512) void attn_kernel(AttnArgs a) {
  using L = AttnLds<T, HD>;
  constexpr int E = L::E;
  constexpr int NQV = HD / (4 * E);   // 16-byte vectors per lane along hd
  constexpr int DT = HD / 16;         // 16-wide dim tiles of O^T
  constexpr int VPR = HD / E;         // 16-byte vectors per K/V row
  constexpr int UB = 4;               // items per thread per load round
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nthr = blockDim.x;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int per = a.H / a.G;          // query heads per K/V head
  const int hpw = per / a.hsplit;     // of them in this workgroup (= waves)
  const int QT = (a.n + 15) / 16;
  // workgroup i runs on XCD i % 8: unit (i % 8) * (grid / 8) + i / 8 puts
  // consecutive units on one XCD (the grid is padded to a multiple of 8)
  const int units = a.B * QT * a.G * a.hsplit * a.kv_split;
  int u = (int)(blockIdx.x % 8u) * (int)(gridDim.x / 8u) + (int)(blockIdx.x / 8u);
  if (u >= units) return;
  const int qh = u % (QT * a.hsplit);
  u /= QT * a.hsplit;
  const int qt = qh / a.hsplit, hs = qh - qt * a.hsplit;
  const int split = u % a.kv_split;
  u /= a.kv_split;
  const int g = u % a.G;
  const int b = u / a.G;
  const int h = g * per + hs * hpw + wave;

  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nbp = (npre + 31) / 32, nbs = (nself + 31) / 32;
  const int jbeg = split * a.key_chunk;
  const int nblk = min(nbp + nbs, jbeg + a.key_chunk) - jbeg;

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

  // key `kr` of block jb of this split: source row pointers, false if past the end
  auto src = [&](int jb, int kr, const T*& kp, const T*& vp) -> bool {
    const int j = jbeg + jb;
    const bool pre = j < nbp;
    const int key = (pre ? j : j - nbp) * 32 + kr;
    if (key >= (pre ? npre : nself)) return false;
    kp = pre ? kc + (size_t)key * HD : ksf + (size_t)key * a.ldkv;
    vp = pre ? vc + (size_t)key * HD : vsf + (size_t)key * a.ldkv;
    return true;
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
  // bf16 V^T reads: byte offset of this lane's 8-byte block for dim tiles d
  // with d % 4 == q (row 8 g4 + r16/4, dims 16 d + 4 (r16 % 4), swizzled)
  int vtr[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    vtr[q] = (8 * g4 + (r16 >> 2)) * HD * 2 + (((2 * q + ((r16 & 3) >> 1)) ^ (2 * (r16 >> 2))) * 16) + (r16 & 1) * 8;

  for (int c0 = 0; c0 < nblk; c0 += KB_MAX) {
    const int cb = min(KB_MAX, nblk - c0);
    if (c0 > 0) __syncthreads();   // the previous chunk's LDS reads are done
    // Stage blocks c0 .. c0+cb-1 of the split into LDS slots 0 .. cb-1.  K item
    // i: vector i % VPR of key row (i / VPR) % 32 of slot i / (32 VPR).  bf16 V
    // items are the same (row-major, swizzled); fp32 V item i is vector
    // i / 16 % VPR of the key pair i % 16, slot i / (16 VPR), written as one
    // 2-element column of V^T.  Keys past the end are zero (no NaN from
    // unwritten LDS).
    const int nk = cb * 32 * VPR;
    if constexpr (E == 8) {
      for (int base = threadIdx.x; base < nk; base += UB * nthr) {
        uint4 kr4[UB], vr4[UB];
#pragma unroll
        for (int q = 0; q < UB; ++q) {
          const int i = base + q * nthr;
          kr4[q] = make_uint4(0, 0, 0, 0);
          vr4[q] = make_uint4(0, 0, 0, 0);
          const T *kp, *vp;
          if (i < nk) {
            const int jb = i / (32 * VPR), r = i - jb * 32 * VPR;
            const int kr = r / VPR, cv = r - kr * VPR;
            if (src(c0 + jb, kr, kp, vp)) {
              kr4[q] = ldg16(kp + cv * E);
              vr4[q] = ldg16(vp + cv * E);
            }
          }
        }
#pragma unroll
        for (int q = 0; q < UB; ++q) {
          const int i = base + q * nthr;
          if (i < nk) {
            const int jb = i / (32 * VPR), r = i - jb * 32 * VPR;
            const int kr = r / VPR, cv = r - kr * VPR;
            T* kl = reinterpret_cast<T*>(smem + jb * L::BUF);
            *reinterpret_cast<uint4*>(kl + kr * L::KP + cv * E) = kr4[q];
            unsigned char* vl = smem + jb * L::BUF + L::KBYTES;
            *reinterpret_cast<uint4*>(vl + (size_t)kr * HD * 2 + (cv ^ (2 * (kr & 3))) * 16) = vr4[q];
          }
        }
      }
    } else {
    const int nv = cb * 16 * VPR;
    for (int base = threadIdx.x; base < nk; base += UB * nthr) {
      uint4 kr4[UB], v0[UB], v1[UB];
#pragma unroll
      for (int q = 0; q < UB; ++q) {
        const int i = base + q * nthr;
        kr4[q] = make_uint4(0, 0, 0, 0);
        v0[q] = make_uint4(0, 0, 0, 0);
        v1[q] = make_uint4(0, 0, 0, 0);
        const T *kp, *vp;
        if (i < nk) {
          const int jb = i / (32 * VPR), r = i - jb * 32 * VPR;
          const int kr = r / VPR, cv = r - kr * VPR;
          if (src(c0 + jb, kr, kp, vp)) kr4[q] = ldg16(kp + cv * E);
        }
        if (i < nv) {
          const int jb = i / (16 * VPR), r = i - jb * 16 * VPR;
          const int kp2 = r & 15, cv = r >> 4;
          if (src(c0 + jb, 2 * kp2, kp, vp)) v0[q] = ldg16(vp + cv * E);
          if (src(c0 + jb, 2 * kp2 + 1, kp, vp)) v1[q] = ldg16(vp + cv * E);
        }
      }
#pragma unroll
      for (int q = 0; q < UB; ++q) {
        const int i = base + q * nthr;
        if (i < nk) {
          const int jb = i / (32 * VPR), r = i - jb * 32 * VPR;
          const int kr = r / VPR, cv = r - kr * VPR;
          T* kl = reinterpret_cast<T*>(smem + jb * L::BUF);
          *reinterpret_cast<uint4*>(kl + kr * L::KP + cv * E) = kr4[q];
        }
        if (i < nv) {
          const int jb = i / (16 * VPR), r = i - jb * 16 * VPR;
          const int kp2 = r & 15, cv = r >> 4;
          T* vl = reinterpret_cast<T*>(smem + jb * L::BUF + L::KBYTES);
          const uint32_t a4[4] = {v0[q].x, v0[q].y, v0[q].z, v0[q].w};
          const uint32_t b4[4] = {v1[q].x, v1[q].y, v1[q].z, v1[q].w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            *reinterpret_cast<uint2*>(vl + (cv * 4 + e) * L::VP + 2 * kp2) = make_uint2(a4[e], b4[e]);
        }
      }
    }
    }
    __syncthreads();

    for (int jb = 0; jb < cb; ++jb) {
      const int j = jbeg + c0 + jb;
      const int cnt = j < nbp ? min(32, npre - j * 32) : min(32, nself - (j - nbp) * 32);
      const T* kl = reinterpret_cast<const T*>(smem + jb * L::BUF);
      const T* vl = reinterpret_cast<const T*>(smem + jb * L::BUF + L::KBYTES);

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
      // lane holds keys 8*g4 + 4t + i for query r16; causal: action key
      // (j - nbp) * 32 + kr is visible to query qrow when it is <= qrow
      const int lim = (a.causal && j >= nbp) ? min(cnt, qrow - (j - nbp) * 32 + 1) : cnt;
      float bmax = -INFINITY;
      float p[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kr = 8 * g4 + 4 * t + i;
          const float v = (kr < lim) ? s[t][i] * sc : -INFINITY;
          p[4 * t + i] = v;
          bmax = fmaxf(bmax, v);
        }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
      const float mnew = fmaxf(mrun, bmax);
      // a query with no visible key so far (causal mask) keeps weight 0
      const float mref = mnew == -INFINITY ? 0.0f : mnew;
      const float corr = exp2f(mrun - mref);
      float psum = 0.0f;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        p[k] = exp2f(p[k] - mref);
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
        // A = V^T (dims 16 d + r16, keys 8 g4 .. + 7) from two transposing
        // reads of the row-major V block (see attn_tile)
        typedef short v4s_t __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) v4s_t lds_v4s;
        const unsigned char* vbase = reinterpret_cast<const unsigned char*>(vl);
#pragma unroll
        for (int d = 0; d < DT; ++d) {
          const unsigned char* ap = vbase + vtr[d & 3] + 128 * (d >> 2);
          const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap));
          const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap + 4 * HD * 2));
          const uint4 va = make_uint4(((uint32_t)(uint16_t)lo[0]) | ((uint32_t)(uint16_t)lo[1] << 16),
                                      ((uint32_t)(uint16_t)lo[2]) | ((uint32_t)(uint16_t)lo[3] << 16),
                                      ((uint32_t)(uint16_t)hi[0]) | ((uint32_t)(uint16_t)hi[1] << 16),
                                      ((uint32_t)(uint16_t)hi[2]) | ((uint32_t)(uint16_t)hi[3] << 16));
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
    }
  }

  // Lane holds O^T[dim = 16d + 4*g4 + i][query r16].
  if (qrow >= a.n) return;
  const float inv = lrun > 0.0f ? 1.0f / lrun : 0.0f;
  // the lane's 4 consecutive dims of each 16-dim tile go out as one store
  auto put4 = [&](T* dst, const f32x4& v) {
    if constexpr (E == 8) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
    } else {
      *reinterpret_cast<float4*>(dst) = make_float4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
    }
  };
  if (a.kv_split == 1) {
    T* op = reinterpret_cast<T*>(a.o) + (size_t)(b * a.n + qrow) * a.ldo + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d) put4(op + d * 16 + 4 * g4, o[d]);
    return;
  }
  // partial: normalised by its own sum, plus (max, sum)
  const int rows = a.B * a.n, dq = a.H * HD;
  T* pp = reinterpret_cast<T*>(a.part) + ((size_t)split * rows + b * a.n + qrow) * dq + h * HD;
#pragma unroll
  for (int d = 0; d < DT; ++d) put4(pp + d * 16 + 4 * g4, o[d]);
  if (g4 == 0) {
    float* st = a.stats + (((size_t)split * rows + b * a.n + qrow) * a.H + h) * 2;
    st[0] = mrun;
    st[1] = lrun;
  }
}

// O[m][h] = sum_s w_s O_s / sum_s w_s with w_s = l_s * 2^(m_s - max_s m_s).
// Q lanes per output vector (16 bytes of one row): lane q of the group merges
// splits q, q + Q, ... (at most MB) in one online pass (running max, rescaled
// sums) with all its loads issued at once, and the group's partial results
// are combined through lane shuffles.  Q = 4 for more than 4 splits (up to
// 64), else Q = 1, so that no lane of a short merge idles.
template <typename T, int MERGE_Q, int MERGE_MB>
__global__ __launch_bounds__(64) void attn_merge_kernel(AttnArgs a) {
  constexpr int E = ElemTraits<T>::E;
  constexpr int VPW = 64 / MERGE_Q;   // vectors per wave
  const int rows = a.B * a.n, dq = a.H * a.hd;
  const int cblocks = (dq + VPW * E - 1) / (VPW * E);
  const int m = blockIdx.x / cblocks;
  const int qt = threadIdx.x & (MERGE_Q - 1);
  const int c = ((blockIdx.x - m * cblocks) * VPW + threadIdx.x / MERGE_Q) * E;
  const bool live = c < dq;           // every lane stays for the shuffles
  const int h = live ? c / a.hd : 0;
  const int S = a.kv_split, H = a.H;
  const T* part = reinterpret_cast<const T*>(a.part);
  uint4 v[MERGE_MB];
  float2 st[MERGE_MB];
#pragma unroll
  for (int j = 0; j < MERGE_MB; ++j) {
    const int sp = qt + MERGE_Q * j;
    const bool ok = live && sp < S;
    st[j] = ok ? *reinterpret_cast<const float2*>(a.stats + (((size_t)sp * rows + m) * H + h) * 2)
               : make_float2(-INFINITY, 0.0f);
    v[j] = ok ? ldg16(part + ((size_t)sp * rows + m) * dq + c) : make_uint4(0, 0, 0, 0);
  }
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  float mx = -INFINITY, tot = 0.0f;
#pragma unroll
  for (int j = 0; j < MERGE_MB; ++j) {
    if (st[j].y <= 0.0f) continue;     // absent split, or one without keys
    const float mnew = fmaxf(mx, st[j].x);
    const float corr = exp2f(mx - mnew);
    const float w = st[j].y * exp2f(st[j].x - mnew);
    float f[E];
    unpack16(v[j], f, T());
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = acc[e] * corr + w * f[e];
    tot = tot * corr + w;
    mx = mnew;
  }
#pragma unroll
  for (int sh = 1; sh < MERGE_Q; sh <<= 1) {
    const float mo = __shfl_xor(mx, sh, 64), to = __shfl_xor(tot, sh, 64);
    const float mn = fmaxf(mx, mo);
    const float cs = tot > 0.0f ? exp2f(mx - mn) : 0.0f, co = to > 0.0f ? exp2f(mo - mn) : 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = acc[e] * cs + __shfl_xor(acc[e], sh, 64) * co;
    tot = tot * cs + to * co;
    mx = mn;
  }
  if (!live || qt != 0) return;
  const float inv = tot > 0.0f ? 1.0f / tot : 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] *= inv;
  stg16(reinterpret_cast<T*>(a.o) + (size_t)m * a.ldo + c, pack16(acc, T()));
}

template <typename T>
hipError_t launch_merge(const AttnArgs& a, hipStream_t s) {
  constexpr int E = ElemTraits<T>::E;
  const int dq = a.H * a.hd, rows = a.B * a.n;
  if (a.kv_split <= 4) {
    const int cblocks = (dq + 64 * E - 1) / (64 * E);
    hipLaunchKernelGGL((attn_merge_kernel<T, 1, 4>), dim3(rows * cblocks), dim3(64), 0, s, a);
  } else {
    const int cblocks = (dq + 16 * E - 1) / (16 * E);
    hipLaunchKernelGGL((attn_merge_kernel<T, 4, 16>), dim3(rows * cblocks), dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s, int which) {
  const int QT = (a.n + 15) / 16;
  const int units = a.B * QT * a.G * a.hsplit * a.kv_split;
  if (units <= 0) return hipSuccess;
  const int grid = (units + 7) / 8 * 8;   // multiple of 8: XCD-aware unit numbering
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, HD>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  if (a.hsplit < 1 || (a.H / a.G) % a.hsplit) return hipErrorInvalidValue;
  const int threads = 64 * (a.H / a.G / a.hsplit);
  using L = AttnLds<T, HD>;
  if (a.key_chunk < 1) return hipErrorInvalidValue;
  const size_t lds = (size_t)(a.key_chunk < KB_MAX ? a.key_chunk : KB_MAX) * L::BUF;
  if (which != 2) {
    hipLaunchKernelGGL((attn_kernel<T, HD>), dim3(grid), dim3(threads), lds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (which == 1 || a.kv_split == 1) return hipSuccess;
  return launch_merge<T>(a, s);
}


// ---------------------------------------------------------------------------
// attn_tile -- large query counts per K/V head (batched requests).  The query
// heads that share K/V head g are flattened into rows (head, query) of one
// group: row R = hh * n + t is query t of head g*per + hh.  A workgroup of 8
// waves (two per SIMD, so one wave's LDS and memory waits hide behind the
// other's MFMAs) takes 128 such rows, 16 per wave, and loops over the split's
// keys in blocks of 64, so every K/V byte staged in LDS serves 128 rows.  Per
// block, in LDS:
//   K   [64 keys][HD]   16-byte chunk c of key k at slot c ^ f(k),
//                       f(k) = (k & 3) | ((k >> 1) & 4)
//   V   [64 keys][HD]   16-byte chunk c of key k at slot c ^ 2 (k % 4)
// Both arrive by direct-to-LDS loads (one wave instruction = 64 slots of
// consecutive rows).  K rows are the A operand of S^T; the XOR gives the 8
// rows one operand load reads per bank cycle (keys 8 (r/4) + r%4 of the
// score-tile permutation) 8 different slots.  The V^T operand of
// O^T += V^T P^T is read with ds_read_b64_tr_b16: within each 16 lanes, lane
// i receives element i % 4 of the 8-byte blocks addressed by lanes i/4,
// i/4 + 4, i/4 + 8 and i/4 + 12.  Lane p of a group therefore addresses key
// row 8 g4 + p/4 (+4 for the second read) at dims 16 d + 4 (p % 4) and gets 4
// consecutive keys of dim 16 d + p; the V swizzle puts the 4 rows one
// 16-lane read touches in 4 disjoint 32-byte bank ranges.
// The next block's loads are in flight while the current block's MFMAs run;
// LDS is double-buffered.  Scores are computed transposed (S^T = K Q^T) with
// the same key permutation as attn_kernel, so a lane's 8 keys of a 32-key half
// are the k slots of its P^T operand in O^T += V^T P^T.  Split outputs use the
// attn_kernel partial format, so attn_merge combines them.

typedef unsigned v4u_t __attribute__((ext_vector_type(4)));
// One wave-wide global_load_lds_dwordx4: lane l's 16 bytes at g land in LDS at
// wave-uniform lds + 16 l.  The compiler does not track it: an explicit
// vmcnt(0) wait (dma_wait_all) before the barrier orders it against the reads.
VLA_DEV void dma16(const void* g, void* lds) {
  typedef __attribute__((address_space(3))) v4u_t lds_v4u;
  const unsigned off = (unsigned)(uintptr_t)(lds_v4u*)lds;
  const unsigned base = __builtin_amdgcn_readfirstlane(off);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(base), "v"(g) : "memory", "m0");
}

// Wait until every load this wave issued has completed, the direct-to-LDS ones
// included: the compiler does not see those (asm) and would not wait for them
// at a barrier by itself.
VLA_DEV void dma_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// V slot swizzle of key k (see attn_tile)
VLA_DEV int vswz(int k) { return 2 * (k & 3); }

constexpr int TQ = 128;   // rows per workgroup
constexpr int TKB = 64;   // keys per block
constexpr int TW = 8;     // waves per workgroup (16 rows each)

template <int HD>
struct TileLds {
  static constexpr int CPR = HD / 8;                          // 16-byte chunks per K row
  static constexpr size_t KB = (size_t)TKB * HD * 2;          // one K block (bf16)
  static constexpr size_t VB = (size_t)TKB * HD * 2;          // one V block
  static constexpr size_t BYTES = 2 * (KB + VB);              // double-buffered
};

template <int HD>
__global__ __launch_bounds__(64 * TW) void attn_tile(AttnArgs a) {
  using L = TileLds<HD>;
  constexpr int CPR = L::CPR;
  constexpr int NQV = HD / 32;                  // k-steps of S^T (16-byte vectors per lane)
  constexpr int DT = HD / 16;                   // dim tiles of O^T
  constexpr int KLD = TKB * CPR / (64 * TW);    // K load instructions per wave and block
  static_assert(KLD >= 1 && KLD * 64 * TW == TKB * CPR, "K staging");
  extern __shared__ __align__(16) unsigned char smem[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int per = a.H / a.G;
  const int nrows = per * a.n;
  const int rt = (nrows + TQ - 1) / TQ;
  const int units = a.B * a.G * rt * a.kv_split;
  int u = (int)(blockIdx.x % 8u) * (int)(gridDim.x / 8u) + (int)(blockIdx.x / 8u);
  if (u >= units) return;
  const int tile = u % rt;
  u /= rt;
  const int split = u % a.kv_split;
  u /= a.kv_split;
  const int g = u % a.G;
  const int b = u / a.G;

  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nkeys = npre + nself;
  const int nblk_all = (nkeys + TKB - 1) / TKB;
  const int jb0 = split * a.key_chunk;
  const int nb = min(nblk_all, jb0 + a.key_chunk) - jb0;

  const bf16_t* kc = reinterpret_cast<const bf16_t*>(a.kc);
  const bf16_t* vc = reinterpret_cast<const bf16_t*>(a.vc);
  if (npre > 0 && kc == nullptr) {
    kc = reinterpret_cast<const bf16_t*>(a.cp->kv_cache) + a.layer_off;
    vc = kc + (size_t)a.B * a.G * a.P * HD;
  }
  kc += ((size_t)b * a.G + g) * a.P * HD;
  vc += ((size_t)b * a.G + g) * a.P * HD;
  const bf16_t* ksf = reinterpret_cast<const bf16_t*>(a.ks) + (size_t)b * a.n * a.ldkv + g * HD;
  const bf16_t* vsf = reinterpret_cast<const bf16_t*>(a.vs) + (size_t)b * a.n * a.ldkv + g * HD;
  // row pointer of key kx < nkeys (prefix rows first)
  auto krow = [&](int kx) -> const bf16_t* {
    return kx < npre ? kc + (size_t)kx * HD : ksf + (size_t)(kx - npre) * a.ldkv;
  };
  auto vrow = [&](int kx) -> const bf16_t* {
    return kx < npre ? vc + (size_t)kx * HD : vsf + (size_t)(kx - npre) * a.ldkv;
  };

  // Q^T fragments of this wave's 16 rows
  const int R = tile * TQ + wave * 16 + r16;
  const bool rok = R < nrows;
  const int tq = rok ? R % a.n : 0;   // the row's action token (query index)
  uint4 qf[NQV];
  {
    const int hh = rok ? R / a.n : 0, t = rok ? R - hh * a.n : 0;
    const bf16_t* qp = reinterpret_cast<const bf16_t*>(a.q) + (size_t)(b * a.n + t) * a.ldq + (g * per + hh) * HD + g4 * (HD / 4);
#pragma unroll
    for (int c = 0; c < NQV; ++c) qf[c] = rok ? ldg16(qp + c * 8) : make_uint4(0, 0, 0, 0);
  }

  // K: wave instruction i fills slots [(TW i + wave) * 64, + 64) of the block:
  // row slot0 / CPR + lane / CPR, slot lane % CPR, which holds k-chunk
  // slot ^ f(row).  Keys past the end read the last key (masked scores).
  // this lane's element offsets inside a block of prefix rows, per instruction
  int koffp[KLD], voffp[KLD];
#pragma unroll
  for (int i = 0; i < KLD; ++i) {
    const int slot0 = (TW * i + wave) * 64;
    const int row = slot0 / CPR + lane / CPR, sl = lane % CPR;
    koffp[i] = row * HD + (sl ^ kswz(row)) * 8;
    voffp[i] = row * HD + (sl ^ vswz(row)) * 8;
  }
  auto kload = [&](int jb, int buf) {
    const int kx0 = (jb0 + jb) * TKB;
    unsigned char* kl = smem + buf * (L::KB + L::VB);
    if (kx0 + TKB <= npre) {  // every row of the block is a prefix row
      const bf16_t* base = kc + (size_t)kx0 * HD;
#pragma unroll
      for (int i = 0; i < KLD; ++i) dma16(base + koffp[i], kl + (size_t)(TW * i + wave) * 64 * 16);
      return;
    }
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int slot0 = (TW * i + wave) * 64;
      const int row = slot0 / CPR + lane / CPR, sl = lane % CPR;
      dma16(krow(min(kx0 + row, nkeys - 1)) + (sl ^ kswz(row)) * 8, kl + (size_t)slot0 * 16);
    }
  };
  // V: the same slots per lane as K, with the chunk swizzle 2 (row % 4).
  // Keys past the end read the last key; their probabilities are exactly
  // zero (masked scores), so they add nothing.
  auto vload = [&](int jb, int buf) {
    const int kx0 = (jb0 + jb) * TKB;
    unsigned char* vl = smem + buf * (L::KB + L::VB) + L::KB;
    if (kx0 + TKB <= npre) {
      const bf16_t* base = vc + (size_t)kx0 * HD;
#pragma unroll
      for (int i = 0; i < KLD; ++i) dma16(base + voffp[i], vl + (size_t)(TW * i + wave) * 64 * 16);
      return;
    }
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int slot0 = (TW * i + wave) * 64;
      const int row = slot0 / CPR + lane / CPR, sl = lane % CPR;
      dma16(vrow(min(kx0 + row, nkeys - 1)) + (sl ^ vswz(row)) * 8, vl + (size_t)slot0 * 16);
    }
  };

  // LDS operand slots of this lane.  Score-tile row r16 is key
  // 32 kk + 4 t + 8 (r16/4) + r16%4, whose swizzle f(key) = r16 % 8 for every
  // kk and t; V^T row d*16 + r16 likewise has swizzle r16 % 8.
  int kslot[NQV];
  {
    const int key0 = 8 * (r16 >> 2) + (r16 & 3), f = r16 & 7;
#pragma unroll
    for (int c = 0; c < NQV; ++c) kslot[c] = key0 * CPR + ((g4 * NQV + c) ^ f);
  }
  // V^T reads: lane p = r16 of group g4 addresses row 8 g4 + p/4 (+4, +32 kk)
  // at dims 16 d + 4 (p % 4): chunk 2 d + (p % 4)/2, swizzled by the row's
  // 2 (row % 4) = 2 (p / 4), byte 8 (p % 2) within it.  vb[q] is the byte
  // offset for dim tiles with d % 4 == q; tile d adds 128 (d / 4).
  int vb[4];
  {
    const int q4 = r16 >> 2;
    const int rowb = (8 * g4 + q4) * HD * 2;
#pragma unroll
    for (int q = 0; q < 4; ++q) vb[q] = rowb + (((2 * q + ((r16 & 3) >> 1)) ^ (2 * q4)) * 16) + (r16 & 1) * 8;
  }

  f32x4 o[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
  const float sc = a.scale * kLog2e;

  kload(0, 0);
  vload(0, 0);
  dma_wait_all();
  __syncthreads();
  for (int jb = 0; jb < nb; ++jb) {
    const int buf = jb & 1;
    // buffer buf ^ 1 was last read in the previous block, which ended with a barrier
    if (jb + 1 < nb) {
      kload(jb + 1, buf ^ 1);
      vload(jb + 1, buf ^ 1);
    }
    const uint4* kl = reinterpret_cast<const uint4*>(smem + buf * (L::KB + L::VB));
    const uint4* vl = reinterpret_cast<const uint4*>(smem + buf * (L::KB + L::VB) + L::KB);
    const int kvalid = min(TKB, nkeys - (jb0 + jb) * TKB);

    // S^T for both 32-key halves: tile t row rho = key 32 kk + 8 (rho/4) + 4 t + rho%4;
    // the four tiles' accumulation chains are interleaved
    f32x4 s[2][2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int t = 0; t < 2; ++t) s[kk][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NQV; ++c)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int t = 0; t < 2; ++t) mma16(s[kk][t], kl[kslot[c] + (kk * 32 + 4 * t) * CPR], qf[c], bf16_t());
    // online softmax; lane keys: 32 kk + 8 g4 + 4 t + i
    float p[2][8];
    float bmax = -INFINITY;
    const int kx0 = (jb0 + jb) * TKB;
    if (kvalid == TKB && !(a.causal && kx0 + TKB > npre)) {  // full block, no causal keys: no mask
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            p[kk][4 * t + i] = s[kk][t][i] * sc;
            bmax = fmaxf(bmax, p[kk][4 * t + i]);
          }
    } else {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kk * 32 + 8 * g4 + 4 * t + i;
            // causal: action key kx0 + key - npre is visible to query tq when <= tq
            const bool vis = key < kvalid && (!a.causal || kx0 + key - npre <= tq);
            const float v = vis ? s[kk][t][i] * sc : -INFINITY;
            p[kk][4 * t + i] = v;
            bmax = fmaxf(bmax, v);
          }
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    // The reference max moves only when a score exceeds it by more than 2^8:
    // exponentials stay below 256 and most blocks skip rescaling O.
    const bool move = bmax > mrun + 8.0f;
    const float mnew = move ? bmax : mrun;
    const float corr = move ? exp2f(mrun - mnew) : 1.0f;
    const float mref = mnew == -INFINITY ? 0.0f : mnew;   // no visible key yet (causal): weight 0
    float psum = 0.f;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[kk][e] = exp2f(p[kk][e] - mref);
        psum += p[kk][e];
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    lrun = lrun * corr + psum;
    mrun = mnew;
    if (__any(move)) {
#pragma unroll
      for (int d = 0; d < DT; ++d) o[d] *= corr;
    }
    uint4 pb[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      pb[kk] = make_uint4(pack_bf16x2(p[kk][0], p[kk][1]), pack_bf16x2(p[kk][2], p[kk][3]),
                          pack_bf16x2(p[kk][4], p[kk][5]), pack_bf16x2(p[kk][6], p[kk][7]));
    // O^T += V^T P^T: A = V^T (dims 16 d .. + 15, keys 32 kk + 8 g4 .. + 7) from
    // two transposing reads of 4 keys each
    {
      typedef short v4s_t __attribute__((ext_vector_type(4)));
      typedef __attribute__((address_space(3))) v4s_t lds_v4s;
      const unsigned char* vbase = reinterpret_cast<const unsigned char*>(vl);
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const unsigned char* ap = vbase + vb[d & 3] + 128 * (d >> 2) + kk * 32 * HD * 2;
          const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap));
          const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap + 4 * HD * 2));
          const uint4 va = make_uint4(((uint32_t)(uint16_t)lo[0]) | ((uint32_t)(uint16_t)lo[1] << 16),
                                      ((uint32_t)(uint16_t)lo[2]) | ((uint32_t)(uint16_t)lo[3] << 16),
                                      ((uint32_t)(uint16_t)hi[0]) | ((uint32_t)(uint16_t)hi[1] << 16),
                                      ((uint32_t)(uint16_t)hi[2]) | ((uint32_t)(uint16_t)hi[3] << 16));
          mma16(o[d], va, pb[kk], bf16_t());
        }
    }
    dma_wait_all();   // the K / V loads of block jb + 1 have landed (this wave's) ...
    __syncthreads();  // ... and every wave's
  }

  // lane holds O^T[dim 16 d + 4 g4 + i][row R]
  if (!rok) return;
  const int rows = a.B * a.n, dq = a.H * HD;
  const int hh = R / a.n, t = R - hh * a.n, h = g * per + hh;
  const float inv = lrun > 0.f ? 1.f / lrun : 0.f;
  bf16_t* dst;
  if (a.kv_split == 1) {
    dst = reinterpret_cast<bf16_t*>(a.o) + (size_t)(b * a.n + t) * a.ldo + h * HD;
  } else {
    dst = reinterpret_cast<bf16_t*>(a.part) + ((size_t)split * rows + b * a.n + t) * dq + h * HD;
    if (g4 == 0) {
      float* st = a.stats + (((size_t)split * rows + b * a.n + t) * a.H + h) * 2;
      st[0] = mrun;
      st[1] = lrun;
    }
  }
#pragma unroll
  for (int d = 0; d < DT; ++d)
    *reinterpret_cast<uint2*>(dst + d * 16 + 4 * g4) =
        make_uint2(pack_bf16x2(o[d][0] * inv, o[d][1] * inv), pack_bf16x2(o[d][2] * inv, o[d][3] * inv));
}

template <int HD>
hipError_t launch_tile_hd(const AttnArgs& a, hipStream_t s, int which) {
  const int per = a.H / a.G;
  const int rt = (per * a.n + TQ - 1) / TQ;
  const int units = a.B * a.G * rt * a.kv_split;
  if (units <= 0) return hipSuccess;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_tile<HD>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  if (which != 2) {
    hipLaunchKernelGGL((attn_tile<HD>), dim3((units + 7) / 8 * 8), dim3(64 * TW), TileLds<HD>::BYTES, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (which == 1 || a.kv_split == 1) return hipSuccess;
  return launch_merge<bf16_t>(a, s);
}

}  // namespace

// Keys per split in 32-key blocks (at most KB_MAX), the number of splits, and
// the workspace.  By default the splits target about 112 workgroups.
// The tiled kernel: bf16, head_dim 64 / 128 / 256, and enough rows per K/V
// head (per * n) and keys to fill its 128-row, 64-key tiles.  Key splits aim
// at about one workgroup per compute unit.
bool attention_tile_eligible(int et, const AttnArgs& a) {
  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int row_tiles = a.B * a.G * (((a.H / a.G) * a.n + TQ - 1) / TQ);
  // below ~16 row tiles (e.g. one request of 50-100 action tokens) the
  // 16-query kernel's finer split of the keys is faster
  return et == ET_BF16 && (a.hd == 64 || a.hd == 128 || a.hd == 256) && row_tiles >= 16 &&
         npre + nself >= 4 * TKB;
}

void attention_tile_split(AttnArgs& a, int want_splits) {
  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nblk = (npre + nself + TKB - 1) / TKB;
  const int rt = ((a.H / a.G) * a.n + TQ - 1) / TQ;
  const int base = a.B * a.G * rt;
  int s = want_splits > 0 ? want_splits : (256 + base / 2) / base;
  s = s < 1 ? 1 : (s > nblk ? nblk : s);
  if (s > 64) s = 64;
  int kc = (nblk + s - 1) / s;
  if (kc < (nblk + 63) / 64) kc = (nblk + 63) / 64;  // at most 64 splits
  a.tiled = 1;
  a.hsplit = 1;
  a.key_chunk = kc;
  a.kv_split = (nblk + kc - 1) / kc;
}

void attention_split(AttnArgs& a, int want_splits, int want_hsplit) {
  a.tiled = 0;
  const int npre = (a.mode == 0) ? 0 : a.P;
  const int nself = (a.mode == 1) ? 0 : a.n;
  const int nblocks = (npre + 31) / 32 + (nself + 31) / 32;
  const int QT = (a.n + 15) / 16;
  const int per = a.H / a.G;
  // Heads per workgroup: each workgroup reads Q and writes O of its heads for
  // its query tile once per key split, so large groups are split until each
  // workgroup holds at most 4 heads.
  int hs = want_hsplit;
  if (hs <= 0) {
    hs = 1;
    while (per / hs > 4 && per % (2 * hs) == 0) hs *= 2;
  }
  if (hs < 1 || per % hs) hs = 1;
  a.hsplit = hs;
  int s = want_splits;
  if (s <= 0) {
    // About 112 workgroups: the merge reads every split's partial output, so
    // past half the chip more splits cost the merge more than they save in
    // the key loop (pi0 shape: 14 splits beat 28 by 0.5 us per layer).
    const int base = a.B * QT * a.G * hs;
    s = (112 + base - 1) / base;
  }
  // two key blocks or fewer: one split, no merge launch (measured faster)
  if (want_splits <= 0 && nblocks <= 2) s = 1;
  s = s < 1 ? 1 : (s > nblocks ? nblocks : s);
  int kc = (nblocks + s - 1) / s;                            // blocks per split
  kc = kc < (nblocks + 63) / 64 ? (nblocks + 63) / 64 : kc;  // at most 64 splits
  if (want_splits <= 0 && kc > KB_MAX) {
    // Splits of at most KB_MAX blocks run without a chunk loop; past about
    // 1024 workgroups (large batches) the grid keeps that size instead and
    // each split loops over its chunks, which also bounds the merge traffic.
    const int base = a.B * QT * a.G * hs;
    const int s_flat = (nblocks + KB_MAX - 1) / KB_MAX;
    if ((long long)base * s_flat <= 1024) {
      kc = KB_MAX;
    } else {
      const int s_big = 1024 / base > 1 ? 1024 / base : 1;
      kc = (nblocks + s_big - 1) / s_big;
    }
  }
  a.key_chunk = kc;
  a.kv_split = (nblocks + kc - 1) / kc;
}

int attention_max_blocks() { return 1024; }   // 32768 keys (no kernel limit; bounds the workspace)

size_t attention_part_bytes(int et, const AttnArgs& a) {
  if (a.kv_split <= 1) return 0;
  return (size_t)a.kv_split * a.B * a.n * a.H * a.hd * (et == ET_BF16 ? 2 : 4);
}

size_t attention_stats_bytes(const AttnArgs& a) {
  if (a.kv_split <= 1) return 0;
  return (size_t)a.kv_split * a.B * a.n * a.H * 2 * sizeof(float);
}

hipError_t launch_attention(int et, const AttnArgs& a, hipStream_t s, int which) {
  if (a.H % a.G != 0 || a.H / a.G > 8 || a.H > 32 || a.kv_split > 64 || a.kv_split < 1) return hipErrorInvalidValue;
  if (a.tiled) {
    if (et != ET_BF16 || a.key_chunk < 1) return hipErrorInvalidValue;
    switch (a.hd) {
      case 64: return launch_tile_hd<64>(a, s, which);
      case 128: return launch_tile_hd<128>(a, s, which);
      case 256: return launch_tile_hd<256>(a, s, which);
    }
    return hipErrorInvalidValue;
  }
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

// Ternary-weight x int8-activation GEMM (W2A8) on the int8 MFMA units.
//
// Weights arrive packed 2 bits each ([N][K/4] bytes, code w+1 of w[n][4j+i] in
// bits 2i..2i+1 of byte j).  Each lane loads 16 packed bytes = 64 consecutive
// weights of one W row and widens them in registers to the codes c = w + 1 in
// {0,1,2} as int8 (byte-permute + masks, no lookup table).  The MFMA then forms
// sum_k q*c, and sum_k q*w = sum_k q*c - sum_k q is recovered with the row sums
// of the activation codes, which the workgroup accumulates while staging X in
// LDS.  All arithmetic is int32 and exact.  A workgroup walks the whole K
// range (its K-slices one after another); only the raw int32 entry splits K
// across workgroups, adding the exact partial sums atomically.  The
// dequantised path with few token rows uses tern_skinny instead.
#include "gemm_epilogue.h"

namespace {

// 16 2-bit codes (one packed dword, natural k order) -> 16 int8 codes.
VLA_DEV i32x4 unpack_codes(uint32_t p) {
  const uint32_t lo = p & 0x33333333u;         // fields 0 and 2 of each byte
  const uint32_t hi = (p >> 2) & 0x33333333u;  // fields 1 and 3 of each byte
  i32x4 r;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t sel = (uint32_t)b | ((uint32_t)(4 + b) << 8) | ((uint32_t)b << 16) | ((uint32_t)(4 + b) << 24);
    const uint32_t t = __builtin_amdgcn_perm(hi, lo, sel);  // [lo_b, hi_b, lo_b, hi_b]
    r[b] = (int)((t & 0x00000303u) | ((t >> 4) & 0x03030000u));
  }
  return r;
}

VLA_DEV int sum_i8x16(uint4 v) {
  int s = 0;
  s = __builtin_amdgcn_sdot4((int)v.x, 0x01010101, s, false);
  s = __builtin_amdgcn_sdot4((int)v.y, 0x01010101, s, false);
  s = __builtin_amdgcn_sdot4((int)v.z, 0x01010101, s, false);
  s = __builtin_amdgcn_sdot4((int)v.w, 0x01010101, s, false);
  return s;
}

// Requires K % 64 == 0 (16-byte aligned packed rows).
template <int MS, int NSUB, int NC>
__global__ __launch_bounds__(256) void tern_kernel(TernArgs a) {
  constexpr int KC = 256;  // 4 lane groups x 64 k
  constexpr int KS = NC * KC;
  constexpr int MT = 16 * MS;
  constexpr int NT = 64 * NSUB;
  constexpr int PITCH = KS + 16;

  extern __shared__ __align__(16) unsigned char smem[];
  int8_t* xs = reinterpret_cast<int8_t*>(smem);
  int* rsum_s = reinterpret_cast<int*>(smem + (size_t)MT * PITCH);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int KB = K / 4;

  int unit = blockIdx.x;
  const int split = unit % a.nsplit;
  unit /= a.nsplit;
  const int ntile = unit % a.n_tiles;
  const int mtile = unit / a.n_tiles;
  const int m0 = mtile * MT;
  const int k0 = split * KS;
  const int kend = min(K, k0 + KS);
  const int nw0 = ntile * NT + wave * 16 * NSUB;

  i32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = i32x4{0, 0, 0, 0};
  if (tid < MT) rsum_s[tid] = 0;

  // K-slices of this split, one after another inside the workgroup
  const int kstop = (a.nsplit > 1) ? kend : K;
  for (int ks0 = k0; ks0 < kstop; ks0 += KS) {
    const int send = min(kstop, ks0 + KS);
    uint4 wreg[NSUB][NC];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int n = nw0 + s * 16 + r16;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int k = ks0 + c * KC + g4 * 64;
        wreg[s][c] = (n < N && k < send) ? ldg16(a.w + (size_t)n * KB + k / 4) : make_uint4(0, 0, 0, 0);
      }
    }
    __syncthreads();  // rsum_s zeroed / previous slice's LDS reads done
    constexpr int VROW = KS / 16;
    for (int i = tid; i < MT * VROW; i += 256) {
      const int row = i / VROW, kv = i - row * VROW;
      const int m = m0 + row, k = ks0 + kv * 16;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (m < M && k < send) {
        v = ldg16(a.x + (size_t)m * K + k);
        atomicAdd(&rsum_s[row], sum_i8x16(v));
      }
      *reinterpret_cast<uint4*>(xs + (size_t)row * PITCH + kv * 16) = v;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (ks0 + c * KC >= send) break;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int8_t* xrow = xs + (size_t)(ms * 16 + r16) * PITCH + c * KC + g4 * 64;
        uint4 xf[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) xf[r] = *reinterpret_cast<const uint4*>(xrow + 16 * r);
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
          const uint32_t pw[4] = {wreg[s][c].x, wreg[s][c].y, wreg[s][c].z, wreg[s][c].w};
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[ms][s] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xf[r]),
                                                               unpack_codes(pw[r]), acc[ms][s], 0, 0, 0);
        }
      }
    }
  }
  __syncthreads();
  // sum q*w = sum q*c - sum q over the K range of this workgroup.
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rs = rsum_s[ms * 16 + g4 * 4 + i];
#pragma unroll
      for (int s = 0; s < NSUB; ++s) acc[ms][s][i] -= rs;
    }

  if (a.nsplit > 1 && a.rscale == nullptr) {
    // Raw int32 output: integer adds are exact and order-free, so the splits
    // accumulate straight into the (zero-filled) output.
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
          const int n = nw0 + s * 16 + r16;
          if (m < M && n < N) atomicAdd(&a.acc_out[(size_t)m * N + n], acc[ms][s][i]);
        }
      }
    return;
  }
  if (a.rscale == nullptr) {
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
          const int n = nw0 + s * 16 + r16;
          if (m < M && n < N) a.acc_out[(size_t)m * N + n] = acc[ms][s][i];
        }
      }
    return;
  }
  // y = acc * (s_w * r_m / 127), with s_w the per-tensor scale of the
  // matrix that W row n belongs to.
  float sw[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    const int n = nw0 + s * 16 + r16;
    sw[s] = (n < N) ? a.wscale[n] : 0.0f;
  }
  f32x4 y[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ms * 16 + g4 * 4 + i;
      const float rm = (m < M) ? a.rscale[m] : 0.0f;
#pragma unroll
      for (int s = 0; s < NSUB; ++s) y[ms][s][i] = (float)acc[ms][s][i] * (sw[s] * rm / 127.0f);
    }
  wave_epilogue<bf16_t, MS, NSUB>(a.e, y, m0, nw0, 0);
}

// Any K % 4 == 0: one thread per output, byte-wise unpacking.
__global__ __launch_bounds__(256) void tern_generic_kernel(const int8_t* x, const uint8_t* w, int M, int N, int K,
                                                           int32_t* out) {
  const long long idx = blockIdx.x * 256LL + threadIdx.x;
  if (idx >= (long long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx - (long long)m * N);
  const uint8_t* wr = w + (size_t)n * (K / 4);
  const int8_t* xr = x + (size_t)m * K;
  int acc = 0;
  for (int j = 0; j < K / 4; ++j) {
    const uint32_t byte = wr[j];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc += (int)xr[4 * j + i] * ((int)((byte >> (2 * i)) & 3u) - 1);
  }
  out[idx] = acc;
}


// 16 2-bit codes -> 16 signed int8 weights w = code - 1: one byte permute per
// dword maps code 0, 1, 2 to 0xFF, 0x00, 0x01.
VLA_DEV i32x4 unpack_signed(uint32_t p) {
  const i32x4 c = unpack_codes(p);
  i32x4 r;
#pragma unroll
  for (int b = 0; b < 4; ++b) r[b] = (int)__builtin_amdgcn_perm(0u, 0x000100FFu, (uint32_t)c[b]);
  return r;
}

// Small-M dequantised W2A8 GEMM.  A workgroup owns 16 * NSUB W rows (a
// gate/up pair of 16-row blocks for GLU) and every token row (M <= 16 MS).
// K is cut into chunks of 256 (4 lane groups x 64); wave w takes chunks w,
// w+4, ..., and issues all W and X loads of up to CPW chunks before their
// MFMAs.  Weights are widened to signed int8, so the MFMA sums q * w
// directly; the four waves' int32 partials are added through LDS (exact),
// then waves 0 .. MS-1 dequantise and run the epilogue of one 16-row subtile.
template <int MS, int NSUB, int CPW>
__global__ __launch_bounds__(256) void tern_skinny(TernArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  i32x4* red = reinterpret_cast<i32x4*>(smem);  // [4][MS][NSUB][64]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N, K = a.K, KB = K / 4;
  const int n0 = blockIdx.x * 16 * NSUB;
  const int nch = (K + 255) / 256;

  i32x4 acc[MS][NSUB];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[ms][s] = i32x4{0, 0, 0, 0};

  for (int c0 = wave; c0 < nch; c0 += 4 * CPW) {
    uint4 wreg[CPW][NSUB];
    uint4 xreg[CPW][MS][4];
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int k = (c0 + 4 * j) * 256 + g4 * 64;   // this lane group's 64 k
      const bool kok = c0 + 4 * j < nch && k < K;
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        const int n = n0 + s * 16 + r16;
        wreg[j][s] = (kok && n < N) ? ldg16(a.w + (size_t)n * KB + k / 4) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int m = ms * 16 + r16;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          xreg[j][ms][r] = (kok && m < M) ? ldg16(a.x + (size_t)m * K + k + 16 * r) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j)
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        const uint32_t pw[4] = {wreg[j][s].x, wreg[j][s].y, wreg[j][s].z, wreg[j][s].w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const i32x4 wv = unpack_signed(pw[r]);
#pragma unroll
          for (int ms = 0; ms < MS; ++ms)
            acc[ms][s] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xreg[j][ms][r]), wv, acc[ms][s], 0, 0, 0);
        }
      }
  }
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) red[((wave * MS + ms) * NSUB + s) * 64 + lane] = acc[ms][s];
  __syncthreads();
  if (wave >= MS || wave * 16 >= M) return;
  const int ms = wave;
  float sw[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    const int n = n0 + s * 16 + r16;
    sw[s] = (n < N) ? a.wscale[n] : 0.0f;
  }
  f32x4 y[1][NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    i32x4 t = red[((0 * MS + ms) * NSUB + s) * 64 + lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) t += red[((w * MS + ms) * NSUB + s) * 64 + lane];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = ms * 16 + g4 * 4 + i;
      const float rm = (m < M) ? a.rscale[m] : 0.0f;
      y[0][s][i] = (float)t[i] * (sw[s] * rm / 127.0f);
    }
  }
  wave_epilogue<bf16_t, 1, NSUB>(a.e, y, ms * 16, n0, 0);
}

// VALU variant of the small-M dequantised W2A8 GEMM (v_dot4_i32_i8 instead of
// the int8 MFMA), for the dot4-versus-matrix-unit comparison: the same packed
// weights and the same exact int32 sums.  A workgroup owns 16 W rows; wave w
// takes rows 4w .. 4w+3, and lane l the 64-wide K chunks l, l + 64, ... of
// every 4096-wide K slice.  The slice's activation codes are staged in LDS
// for 16 token rows at a time (larger M: further passes over W).  A lane
// widens its 4 rows' packed bytes to signed int8 once per chunk and forms the
// 4 x 16 dot products of the chunk with sdot4 (16 per row and token row).
// The 64 lanes' partial sums are added through LDS in lane order.  Output:
// y = acc * s_w * r_m / 127 to e.out (fp32 or bf16, row-major, EPI_STORE).
constexpr int D4_ROWS = 16, D4_RG = 4, D4_MB = 16, D4_KSL = 64 * 64;
constexpr size_t D4_LDS = (size_t)D4_MB * D4_KSL + (size_t)4 * D4_RG * D4_MB * 64 * 4;

__global__ __launch_bounds__(256) void tern_dot4(TernArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  int8_t* xs = reinterpret_cast<int8_t*>(smem);                              // [D4_MB][D4_KSL]
  int* red = reinterpret_cast<int*>(smem + (size_t)D4_MB * D4_KSL);          // [4][D4_RG][D4_MB][64]
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int M = a.M, N = a.N, K = a.K, KB = K / 4;
  const int n0 = blockIdx.x * D4_ROWS + wave * D4_RG;
  for (int m0 = 0; m0 < M; m0 += D4_MB) {
    int acc[D4_RG][D4_MB];
#pragma unroll
    for (int r = 0; r < D4_RG; ++r)
#pragma unroll
      for (int m = 0; m < D4_MB; ++m) acc[r][m] = 0;
    for (int ks = 0; ks < K; ks += D4_KSL) {
      const int k = ks + lane * 64;
      i32x4 wv[D4_RG][4];
#pragma unroll
      for (int r = 0; r < D4_RG; ++r) {
        const int n = n0 + r;
        const uint4 p = (n < N && k < K) ? ldg16(a.w + (size_t)n * KB + k / 4) : make_uint4(0, 0, 0, 0);
        wv[r][0] = unpack_signed(p.x);
        wv[r][1] = unpack_signed(p.y);
        wv[r][2] = unpack_signed(p.z);
        wv[r][3] = unpack_signed(p.w);
      }
      __syncthreads();   // the previous slice's LDS reads are done
      constexpr int VR = D4_KSL / 16;
      for (int i = t; i < D4_MB * VR; i += 256) {
        const int row = i / VR, kv = i - row * VR;
        const int m = m0 + row, kk = ks + kv * 16;
        const uint4 v = (m < M && kk < K) ? ldg16(a.x + (size_t)m * K + kk) : make_uint4(0, 0, 0, 0);
        *reinterpret_cast<uint4*>(xs + (size_t)row * D4_KSL + kv * 16) = v;
      }
      __syncthreads();
      if (k < K) {
#pragma unroll
        for (int m = 0; m < D4_MB; ++m) {
          if (m0 + m >= M) break;
          const uint4* xp = reinterpret_cast<const uint4*>(xs + (size_t)m * D4_KSL + lane * 64);
          uint4 xv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) xv[q] = xp[q];
#pragma unroll
          for (int r = 0; r < D4_RG; ++r) {
            int s = acc[r][m];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              s = __builtin_amdgcn_sdot4((int)xv[q].x, wv[r][q][0], s, false);
              s = __builtin_amdgcn_sdot4((int)xv[q].y, wv[r][q][1], s, false);
              s = __builtin_amdgcn_sdot4((int)xv[q].z, wv[r][q][2], s, false);
              s = __builtin_amdgcn_sdot4((int)xv[q].w, wv[r][q][3], s, false);
            }
            acc[r][m] = s;
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < D4_RG; ++r)
#pragma unroll
      for (int m = 0; m < D4_MB; ++m) red[((wave * D4_RG + r) * D4_MB + m) * 64 + lane] = acc[r][m];
    __syncthreads();
    // 16 rows x 16 token rows: one output per thread
    {
      const int row = t / D4_MB, m = t - row * D4_MB;
      const int w = row / D4_RG, r = row - w * D4_RG;
      const int* src = red + ((w * D4_RG + r) * D4_MB + m) * 64;
      int s = 0;
      for (int j = 0; j < 64; ++j) s += src[j];
      const int n = blockIdx.x * D4_ROWS + row, mm = m0 + m;
      if (n < N && mm < M) {
        const float y = (float)s * (a.wscale[n] * a.rscale[mm] / 127.0f);
        if (a.e.out_f32) reinterpret_cast<float*>(a.e.out)[(size_t)mm * a.e.ldo + n] = y;
        else reinterpret_cast<bf16_t*>(a.e.out)[(size_t)mm * a.e.ldo + n] = f2bf(y);
      }
    }
    __syncthreads();   // red and xs are reused by the next pass
  }
}

template <int MS, int NSUB>
hipError_t skinny_launch(const TernArgs& a, hipStream_t s) {
  constexpr int CPW = MS == 1 ? (NSUB == 1 ? 8 : 4) : (MS == 2 ? 4 : 2);  // <= 256 VGPRs: two waves per SIMD
  const int grid = (a.N + 16 * NSUB - 1) / (16 * NSUB);
  const size_t lds = (size_t)4 * MS * NSUB * 64 * 16;
  hipLaunchKernelGGL((tern_skinny<MS, NSUB, CPW>), dim3(grid), dim3(256), lds, s, a);
  return hipGetLastError();
}

template <int MS, int NSUB, int NC>
hipError_t tern_launch(const TernArgs& a, int units, hipStream_t s) {
  constexpr int MT = 16 * MS;
  const size_t lds = (size_t)MT * (NC * 256 + 16) + (size_t)MT * 4;
  hipLaunchKernelGGL((tern_kernel<MS, NSUB, NC>), dim3(units), dim3(256), lds, s, a);
  return hipGetLastError();
}

template <int MS, int NSUB>
hipError_t tern_nc(int nc, const TernArgs& a, int units, hipStream_t s) {
  switch (nc) {
    case 1: return tern_launch<MS, NSUB, 1>(a, units, s);
    case 2: return tern_launch<MS, NSUB, 2>(a, units, s);
    case 4: return tern_launch<MS, NSUB, 4>(a, units, s);
    case 8: return tern_launch<MS, NSUB, 8>(a, units, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_ternary_dot4(const TernArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.K % 64 != 0 || a.rscale == nullptr || a.e.epi != EPI_STORE) return hipErrorInvalidValue;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&tern_dot4),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)D4_LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int grid = (a.N + D4_ROWS - 1) / D4_ROWS;
  hipLaunchKernelGGL(tern_dot4, dim3(grid), dim3(256), D4_LDS, s, a);
  return hipGetLastError();
}

// ms: m-subtiles (1, 2, 4); nsub 1 or 2 (GLU pairs); nc from a.ks / 256.
namespace {

// ---------------------------------------------------------------------------
// tern_tile: the W2A8 GEMM with many token rows (the backbone prefill and the
// prefix K/V build, M = B * P), where the int8 matrix cores, not the weight
// bytes, set the pace.  A workgroup owns a (32 MS) x 128 output tile; wave w
// owns its columns 32 w .. 32 w + 31 over all of its rows, so each packed
// weight dword is widened by one wave only (widening costs more vector-ALU
// instructions than the MFMAs it feeds).  128-deep K-slices of the activation codes (BM rows x 128 bytes) and of
// the packed weights (128 rows x 32 bytes) stream into a ring of NST LDS
// stages by direct-to-LDS loads, NST - 1 slices ahead of the MFMAs.  Code rows
// are XOR-swizzled (16-byte chunk c of row r at c ^ (r % 8)), weight rows swap
// their two halves every 8 rows, so the operand reads of 16 rows spread over
// the banks.  Right before its MFMA a lane widens its 16 weights (one dword) to
// signed int8, so v_mfma_i32_16x16x64_i8 sums q * w directly (exact int32).
// Requires K % 128 == 0; rows past M or N load a valid row and are not stored.
// NWV waves of 32 columns each: a 128-column tile on four waves, or a
// 256-column one on eight, whose K-slice (codes + weights) then feeds twice
// the MFMAs for 1.2x (MS = 4) the bytes.
template <int MS, int NWV = 4>
struct TRing {
  static constexpr int BM = 32 * MS, BN = 32 * NWV;
  static constexpr int SX = BM * 8;        // 16-byte slots of codes per stage
  static constexpr int SW = BN * 2;        // 16-byte slots of packed weights per stage
  static constexpr int SB = SX + SW;
  // 80 / 48 / 32 KB of LDS (MS = 4 / 2 / 1, four waves): two or more
  // workgroups fit a CU; 96 KB for MS = 4 on eight waves.  Eight stages time
  // the same as four.
  static constexpr int NST = 4;
  static constexpr int LX = SX / (64 * NWV);   // code loads per thread and slice (weights: one)
  static_assert(LX >= 1 && LX * 64 * NWV == SX, "code rows per wave");
};

template <int MS, int NWV = 4>
__global__ __launch_bounds__(64 * NWV) void tern_tile(TernArgs a) {
  using R = TRing<MS, NWV>;
  constexpr int BM = R::BM, BN = R::BN, SX = R::SX, SB = R::SB, NST = R::NST, LX = R::LX, D = NST - 1;
  static_assert((D - 1) * (LX + 1) < 64, "vmcnt range");
  __shared__ v4u ring[NST][SB];
  auto stage = [&](auto j) -> v4u* { return ring[decltype(j)::value]; };
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  constexpr int RS = 2 * MS;               // 16-row subtiles of the tile, all in every wave
  const int M = a.M, N = a.N, K = a.K, KB = K / 4;
  const int per = gridDim.x >> 3;
  const int u = (blockIdx.x & 7) * per + (blockIdx.x >> 3);   // tiles of one W column block stay on one XCD
  const int tiles = a.m_tiles * a.n_tiles;
  if (u >= tiles) return;
  const int ntile = u / a.m_tiles, mtile = u - ntile * a.m_tiles;
  const int m0 = mtile * BM, n0 = ntile * BN;
  const int nsl = K / 128;

  // sources of this lane's slots: codes (instruction i: row (NWV i + wave) * 8 + lane / 8),
  // weights (row wave * 32 + lane / 2, half lane % 2)
  const int8_t* xsrc[LX];
#pragma unroll
  for (int i = 0; i < LX; ++i) {
    const int row = (i * NWV + wave) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    xsrc[i] = a.x + (size_t)min(m0 + row, M - 1) * K + c * 16;
  }
  const int wrow = wave * 32 + (lane >> 1);
  const uint8_t* wsrc = a.w + (size_t)min(n0 + wrow, N - 1) * KB + (((lane & 1) ^ ((wrow >> 3) & 1)) * 16);
  auto issue = [&](auto j, int sl) {
    v4u* b = stage(j);
#pragma unroll
    for (int i = 0; i < LX; ++i) dma16(xsrc[i] + sl * 128, b + (i * NWV + wave) * 64);
    dma16(wsrc + sl * 32, b + SX + wave * 64);
  };

  i32x4 acc[RS][2];
#pragma unroll
  for (int ms = 0; ms < RS; ++ms)
#pragma unroll
    for (int ns = 0; ns < 2; ++ns) acc[ms][ns] = i32x4{0, 0, 0, 0};

  // MFMA kk of a slice: lane group g4 holds k = 64 kk + 16 g4 .. + 15 of both operands
  auto compute = [&](const v4u* b) {
    v4u xf[2][RS];
    uint32_t wp[2][2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int ms = 0; ms < RS; ++ms) {
        const int row = ms * 16 + r16;
        xf[kk][ms] = b[row * 8 + ((kk * 4 + g4) ^ (row & 7))];
      }
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) {
        const int row = wave * 32 + ns * 16 + r16;
        const uint32_t* slot = reinterpret_cast<const uint32_t*>(b + SX + row * 2 + (kk ^ ((row >> 3) & 1)));
        wp[kk][ns] = slot[g4];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) {
        const i32x4 w = unpack_signed(wp[kk][ns]);
#pragma unroll
        for (int ms = 0; ms < RS; ++ms)
          acc[ms][ns] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xf[kk][ms]), w, acc[ms][ns],
                                                               0, 0, 0);
      }
  };

  [&]<int... J>(std::integer_sequence<int, J...>) {
    ((J < nsl ? issue(std::integral_constant<int, J>{}, J) : void()), ...);
  }(std::make_integer_sequence<int, D>{});
  for (int it0 = 0; it0 < nsl; it0 += NST) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      (
          [&] {
            const int it = it0 + J;
            if (it >= nsl) return;
            // slice `it` has landed once at most the D-1 later slices are pending
            if (it + D - 1 < nsl)
              __builtin_amdgcn_s_waitcnt(vm_wait((D - 1) * (LX + 1)));
            else
              __builtin_amdgcn_s_waitcnt(vm_wait(0));
            lds_barrier();
            if (it + D < nsl) issue(std::integral_constant<int, (J + D) % NST>{}, it + D);
            compute(stage(std::integral_constant<int, J>{}));
          }(),
          ...);
    }(std::make_integer_sequence<int, NST>{});
  }

  const int nw = n0 + wave * 32;
  if (a.rscale == nullptr) {   // raw int32 sums
#pragma unroll
    for (int ms = 0; ms < RS; ++ms)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
        for (int ns = 0; ns < 2; ++ns) {
          const int n = nw + ns * 16 + r16;
          if (m < M && n < N) a.acc_out[(size_t)m * N + n] = acc[ms][ns][i];
        }
      }
    return;
  }
  // y = acc * (s_w * r_m / 127) (the dequantisation of the other W2A8 kernels)
  float sw[2];
#pragma unroll
  for (int ns = 0; ns < 2; ++ns) {
    const int n = nw + ns * 16 + r16;
    sw[ns] = (n < N) ? a.wscale[n] : 0.0f;
  }
  f32x4 y[RS][2];
#pragma unroll
  for (int ms = 0; ms < RS; ++ms)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ms * 16 + g4 * 4 + i;
      const float rm = (m < M) ? a.rscale[m] : 0.0f;
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) y[ms][ns][i] = (float)acc[ms][ns][i] * (sw[ns] * rm / 127.0f);
    }
  if (a.e.epi == EPI_RESID) {         // one 16-column subtile at a time
#pragma unroll
    for (int ns = 0; ns < 2; ++ns) {
      f32x4 y1[RS][1];
#pragma unroll
      for (int ms = 0; ms < RS; ++ms) y1[ms][0] = y[ms][ns];
      wave_epilogue<bf16_t, RS, 1>(a.e, y1, m0, nw + 16 * ns, 0);
    }
  } else {                            // GLU: the wave's 32 columns are one gate / up pair of 16-row blocks
    wave_epilogue<bf16_t, RS, 2>(a.e, y, m0, nw, 0);
  }
}

// tern_tile with two wave groups taking alternate K-slices: eight waves, two
// per SIMD, so one wave's LDS and load waits hide behind the other's work,
// while each packed weight dword is still widened by one wave only (wave
// (g, w) owns columns 32 w .. 32 w + 31 of slices 2 p + g).  Slice pairs
// stream into a ring of NPR pairs (each stage laid out as tern_tile's),
// NPR - 1 pairs ahead of the MFMAs.  At the end group 1 hands its int32
// sums to group 0 through LDS (exact), and group 0 runs the epilogue.
template <int MS>
__global__ __launch_bounds__(512) void tern_tile_kg(TernArgs a) {
  using R = TRing<MS, 4>;
  constexpr int BM = R::BM, BN = R::BN, SX = R::SX, SB = R::SB, LX = R::LX;
  constexpr int NPR = 3;                   // slice pairs in the ring
  constexpr int RS = 2 * MS;               // 16-row subtiles of the tile, all in every wave
  __shared__ v4u ring[2 * NPR][SB];
  static_assert((size_t)4 * RS * 2 * 64 <= (size_t)2 * NPR * SB, "reduction buffer");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = wave >> 2, wl = wave & 3;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int M = a.M, N = a.N, K = a.K, KB = K / 4;
  const int per = gridDim.x >> 3;
  const int u = (blockIdx.x & 7) * per + (blockIdx.x >> 3);   // tiles of one W column block stay on one XCD
  const int tiles = a.m_tiles * a.n_tiles;
  if (u >= tiles) return;
  const int ntile = u / a.m_tiles, mtile = u - ntile * a.m_tiles;
  const int m0 = mtile * BM, n0 = ntile * BN;
  const int nsl = K / 128, npair = (nsl + 1) / 2;

  // this wave's slots in its group's slice, as wave wl of tern_tile
  const int8_t* xsrc[LX];
#pragma unroll
  for (int i = 0; i < LX; ++i) {
    const int row = (i * 4 + wl) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    xsrc[i] = a.x + (size_t)min(m0 + row, M - 1) * K + c * 16;
  }
  const int wrow = wl * 32 + (lane >> 1);
  const uint8_t* wsrc = a.w + (size_t)min(n0 + wrow, N - 1) * KB + (((lane & 1) ^ ((wrow >> 3) & 1)) * 16);
  auto mine = [&](int p) { return 2 * p + grp < nsl; };   // this group's slice of pair p exists
  auto issue = [&](int p) {
    if (!mine(p)) return;
    const int sl = 2 * p + grp;
    v4u* b = ring[2 * (p % NPR) + grp];
#pragma unroll
    for (int i = 0; i < LX; ++i) dma16(xsrc[i] + sl * 128, b + (i * 4 + wl) * 64);
    dma16(wsrc + sl * 32, b + SX + wl * 64);
  };

  i32x4 acc[RS][2];
#pragma unroll
  for (int ms = 0; ms < RS; ++ms)
#pragma unroll
    for (int ns = 0; ns < 2; ++ns) acc[ms][ns] = i32x4{0, 0, 0, 0};

  auto compute = [&](const v4u* b) {
    v4u xf[2][RS];
    uint32_t wp[2][2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int ms = 0; ms < RS; ++ms) {
        const int row = ms * 16 + r16;
        xf[kk][ms] = b[row * 8 + ((kk * 4 + g4) ^ (row & 7))];
      }
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) {
        const int row = wl * 32 + ns * 16 + r16;
        const uint32_t* slot = reinterpret_cast<const uint32_t*>(b + SX + row * 2 + (kk ^ ((row >> 3) & 1)));
        wp[kk][ns] = slot[g4];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) {
        const i32x4 w = unpack_signed(wp[kk][ns]);
#pragma unroll
        for (int ms = 0; ms < RS; ++ms)
          acc[ms][ns] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xf[kk][ms]), w, acc[ms][ns],
                                                               0, 0, 0);
      }
  };

  for (int p = 0; p < NPR - 1 && p < npair; ++p) issue(p);
  for (int p = 0; p < npair; ++p) {
    // this wave's slice of pair p has landed once at most its slice of pair
    // p + 1 (issued, if it exists) is pending
    if (p + 1 < npair && mine(p + 1))
      __builtin_amdgcn_s_waitcnt(vm_wait(LX + 1));
    else
      __builtin_amdgcn_s_waitcnt(vm_wait(0));
    lds_barrier();
    // the stages of pair p - 1 are free: refill them with pair p + NPR - 1
    if (p + NPR - 1 < npair) issue(p + NPR - 1);
    if (mine(p)) compute(ring[2 * (p % NPR) + grp]);
  }
  __builtin_amdgcn_s_waitcnt(vm_wait(0));
  lds_barrier();

  // group 1's sums to group 0 (lane-major, conflict free), exact int32
  i32x4* red = reinterpret_cast<i32x4*>(&ring[0][0]);
  if (grp == 1) {
#pragma unroll
    for (int ms = 0; ms < RS; ++ms)
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) red[((wl * RS + ms) * 2 + ns) * 64 + lane] = acc[ms][ns];
  }
  lds_barrier();
  if (grp == 1) return;
#pragma unroll
  for (int ms = 0; ms < RS; ++ms)
#pragma unroll
    for (int ns = 0; ns < 2; ++ns) acc[ms][ns] += red[((wl * RS + ms) * 2 + ns) * 64 + lane];

  const int nw = n0 + wl * 32;
  if (a.rscale == nullptr) {   // raw int32 sums
#pragma unroll
    for (int ms = 0; ms < RS; ++ms)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ms * 16 + g4 * 4 + i;
#pragma unroll
        for (int ns = 0; ns < 2; ++ns) {
          const int n = nw + ns * 16 + r16;
          if (m < M && n < N) a.acc_out[(size_t)m * N + n] = acc[ms][ns][i];
        }
      }
    return;
  }
  float sw[2];
#pragma unroll
  for (int ns = 0; ns < 2; ++ns) {
    const int n = nw + ns * 16 + r16;
    sw[ns] = (n < N) ? a.wscale[n] : 0.0f;
  }
  f32x4 y[RS][2];
#pragma unroll
  for (int ms = 0; ms < RS; ++ms)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ms * 16 + g4 * 4 + i;
      const float rm = (m < M) ? a.rscale[m] : 0.0f;
#pragma unroll
      for (int ns = 0; ns < 2; ++ns) y[ms][ns][i] = (float)acc[ms][ns][i] * (sw[ns] * rm / 127.0f);
    }
  if (a.e.epi == EPI_RESID) {         // one 16-column subtile at a time
#pragma unroll
    for (int ns = 0; ns < 2; ++ns) {
      f32x4 y1[RS][1];
#pragma unroll
      for (int ms = 0; ms < RS; ++ms) y1[ms][0] = y[ms][ns];
      wave_epilogue<bf16_t, RS, 1>(a.e, y1, m0, nw + 16 * ns, 0);
    }
  } else {                            // GLU: the wave's 32 columns are one gate / up pair of 16-row blocks
    wave_epilogue<bf16_t, RS, 2>(a.e, y, m0, nw, 0);
  }
}

template <int MS>
hipError_t tile_kg_launch(const TernArgs& a0, hipStream_t s) {
  TernArgs a = a0;
  a.m_tiles = (a.M + 32 * MS - 1) / (32 * MS);
  a.n_tiles = (a.N + 127) / 128;
  const int tiles = a.m_tiles * a.n_tiles;
  const int grid = (tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((tern_tile_kg<MS>), dim3(grid), dim3(512), 0, s, a);
  return hipGetLastError();
}

template <int MS, int NWV = 4>
hipError_t tile_launch(const TernArgs& a0, hipStream_t s) {
  TernArgs a = a0;
  a.m_tiles = (a.M + 32 * MS - 1) / (32 * MS);
  a.n_tiles = (a.N + 32 * NWV - 1) / (32 * NWV);
  const int tiles = a.m_tiles * a.n_tiles;
  const int grid = (tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((tern_tile<MS, NWV>), dim3(grid), dim3(64 * NWV), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool tern_tile_eligible(int M, int N, int K) { return M >= 128 && N >= 1 && K >= 128 && K % 128 == 0; }

hipError_t launch_ternary_tile(const TernArgs& a, int ms, int waves, int kgroups, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (!tern_tile_eligible(a.M, a.N, a.K) || a.nsplit > 1) return hipErrorInvalidValue;
  switch (ms * 100 + waves * 10 + kgroups) {
    case 141: return tile_launch<1>(a, s);
    case 241: return tile_launch<2>(a, s);
    case 441: return tile_launch<4>(a, s);
    case 281: return tile_launch<2, 8>(a, s);
    case 481: return tile_launch<4, 8>(a, s);
    case 182: return tile_kg_launch<1>(a, s);
    case 282: return tile_kg_launch<2>(a, s);
    case 482: return tile_kg_launch<4>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_ternary_gemm(const TernArgs& a, int ms, int units, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.K % 64 != 0) {
    if (a.rscale != nullptr) return hipErrorInvalidValue;
    const long long total = (long long)a.M * a.N;
    hipLaunchKernelGGL(tern_generic_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a.x, a.w, a.M,
                       a.N, a.K, a.acc_out);
    return hipGetLastError();
  }
  const int nsub = (a.rscale != nullptr && a.e.epi == EPI_GLU) ? 2 : 1;
  if (a.nsplit <= 1 && tern_tile_eligible(a.M, a.N, a.K)) {
    // many token rows: the tiled kernel; 64 x 256 tiles on eight waves when
    // they still fill the device (the wide gate/up shape), else 128-row
    // tiles once they do; below that, 64-row (or, when those would leave
    // half the device idle, 32-row) tiles on eight waves in two K groups
    const long long nt = (a.N + 127) / 128, nt2 = (a.N + 255) / 256;
    const long long t4 = (long long)((a.M + 127) / 128) * nt, t2 = (long long)((a.M + 63) / 64) * nt;
    const long long t28 = (long long)((a.M + 63) / 64) * nt2;
    if (t28 >= 256) return tile_launch<2, 8>(a, s);
    return t4 >= 256 ? tile_launch<4>(a, s) : t2 >= 128 ? tile_kg_launch<2>(a, s) : tile_kg_launch<1>(a, s);
  }
  if (a.rscale != nullptr && a.M <= 64) {  // token rows of the denoise loop: the skinny kernel
    const int sms = a.M <= 16 ? 1 : (a.M <= 32 ? 2 : 4);
    switch (sms * 10 + nsub) {
      case 11: return skinny_launch<1, 1>(a, s);
      case 12: return skinny_launch<1, 2>(a, s);
      case 21: return skinny_launch<2, 1>(a, s);
      case 22: return skinny_launch<2, 2>(a, s);
      case 41: return skinny_launch<4, 1>(a, s);
      case 42: return skinny_launch<4, 2>(a, s);
    }
    return hipErrorInvalidValue;
  }
  const int nc = a.ks / 256;
  switch (ms * 10 + nsub) {
    case 11: return tern_nc<1, 1>(nc, a, units, s);
    case 12: return tern_nc<1, 2>(nc, a, units, s);
    case 21: return tern_nc<2, 1>(nc, a, units, s);
    case 22: return tern_nc<2, 2>(nc, a, units, s);
    case 41: return tern_nc<4, 1>(nc, a, units, s);
    case 42: return tern_nc<4, 2>(nc, a, units, s);
  }
  return hipErrorInvalidValue;
}

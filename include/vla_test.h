/*
 * vla_test.h -- per-kernel entry points of libvla for parity tests.
 *
 * Not part of the product ABI.  Each call validates its arguments like the
 * product calls, runs one kernel of the denoise loop on `stream`, synchronises
 * the stream (test entries allocate and free scratch memory) and returns.
 * All buffers are device pointers, 16-byte aligned.  elem: 0 = fp32, 1 = bf16.
 */
#ifndef VLA_TEST_H_
#define VLA_TEST_H_

#include "vla.h"

#ifdef __cplusplus
extern "C" {
#endif

/* y[M][N] (fp32) = x[M][K] w[N][K]^T on the MFMA GEMMs of the projections.
 * K % 8 == 0 (bf16) or K % 4 == 0 (fp32).  variant: 0 = the runtime's choice,
 * 1 = the wide kernel, 2 = the skinny kernel (VLA_E_UNSUPPORTED if the shape
 * does not fit it), 3 = the tiled kernel with the runtime's tile, 4 = the
 * launch of the residual projections: split-K fp32 partials (the runtime's
 * split and tile), summed into y by the library (VLA_E_UNSUPPORTED for fp32
 * with M > 128; a temporary partial buffer is allocated and freed),
 * 10..14 = the tiled kernel with tile 64x128, 128x128, 256x128, 128x256 or
 * 256x256 (eight waves; needs K % 64 == 0) (VLA_E_UNSUPPORTED unless bf16
 * with M > 128, and for 256x256 with K % 64 != 0). */
vla_status vla_test_gemm(int32_t elem, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                         int32_t variant, float* y, void* stream);

/* Attention of B requests of n action tokens (paper Sec. 3.1: the action head
 * cross-attends to the cached prefix).  mode 0 self (keys = the n tokens),
 * 1 cross (keys = the P cached rows), 2 joint (one softmax over both);
 * mode + 4 (self or joint): the causal variant, query t sees the action keys
 * 0 .. t only (and every prefix row).
 *   q [B*n][H*hd]; k_self, v_self [B*n][G*hd]; k_cache, v_cache [B][G][P][hd];
 *   o [B*n][H*hd]; all in elem.  kv_split: key splits (kv_split % 100) and
 *   query-head groups per K/V head (kv_split / 100); 0 in either part lets
 *   the runtime choose.  kv_split >= 1000 selects the 128-row tiled kernel
 *   (bf16 only) with kv_split - 1000 key splits of 64-key blocks (0 = the
 *   runtime's count). */
vla_status vla_test_attention(int32_t elem, int32_t mode, const void* q, const void* k_self,
                              const void* v_self, const void* k_cache, const void* v_cache, int32_t B,
                              int32_t n, int32_t P, int32_t H, int32_t G, int32_t hd, int32_t kv_split,
                              void* o, void* stream);

/* Per-token absmax int8 quantiser of the W2A8 path: x [M][K] fp32 ->
 * q [M][K] int8, r [M] fp32. */
vla_status vla_test_quantize_i8(const float* x, int32_t M, int32_t K, int8_t* q, float* r, void* stream);

/* The same quantiser on bf16 rows with a row pitch: x [M][ldx] bf16 bits
 * (ldx >= K, K <= 16384) -> q [M][K] int8, r [M] fp32.  Rows whose values
 * fill whole aligned 16-byte vectors take the register-resident kernel,
 * others the looping one; both give the same codes. */
vla_status vla_test_quantize_bf16(const uint16_t* x, int32_t M, int32_t K, int32_t ldx, int8_t* q, float* r,
                                  void* stream);

/* W2A8 linear: quantise x [M][K] fp32 per token, multiply by the packed
 * ternary w [N][K/4] (K % 64 == 0) and dequantise with the per-tensor scale
 * `scale`: y [M][N] fp32 = acc * scale * r_m / 127. */
vla_status vla_test_ternary_linear(const float* x, const uint8_t* w_packed, int32_t M, int32_t N, int32_t K,
                                   float scale, float* y, void* stream);

/* Rotary position embedding in place (the VLA_OPT_ROPE_BASE variant's
 * kernel): x [rows][ld] in elem (0 fp32, 1 bf16), heads h < nheads of hd
 * values from column col0; row r is at position pos0 + r % rows_per_request.
 * With h2 = hd/2 and w_i = base^(-2i/hd), the pair (i, i+h2) of a head turns
 * by pos * w_i (rotate-half form).  hd even, base > 1.  Synchronises. */
vla_status vla_test_rope(int32_t elem, void* x, int32_t rows, int32_t rows_per_request, int32_t ld, int32_t col0,
                         int32_t nheads, int32_t hd, int32_t pos0, float base, void* stream);

/* The W2A8 GEMM alone, on int8 activation codes already quantised, for the
 * comparison of the paper's dot4 instruction path with its matrix-unit path
 * (Sec. 4.5, the utilisation lever: the same ternary weights on dp4a versus the tensor cores; here
 * v_dot4_i32_i8 on the vector ALUs versus v_mfma_i32_16x16x64_i8).
 *   q [M][K] int8 codes, r [M] fp32 per-row absmax, w_packed [N][K/4] (the
 *   2-bit layout of vla_test_ternary_linear), wscale [N] fp32, y [M][N] fp32:
 *   y = (sum_k q w) * wscale[n] * r[m] / 127.  All device pointers, 16-byte
 *   aligned; K % 64 == 0, 64 <= K <= 16384.
 *   variant 0: the library's W2A8 launch (int8 MFMA); 1: the vector-ALU
 *   sdot4 kernel; 2, 3, 4: the many-row tiled kernel with 32-, 64- or
 *   128-row tiles of 128 columns; 5, 6: 64- or 128-row tiles of 256 columns
 *   on eight waves; 7, 8, 9: 32-, 64- or 128-row tiles of 128 columns on
 *   eight waves in two groups taking alternate K-slices (2..9 need M >= 128
 *   and K % 128 == 0).  All sum exactly in int32, so y is identical.
 *   iters >= 1 (at most 10000): the GEMM runs once untimed, then iters times
 *   between two HIP events on `stream`; *us_per_launch (host, may be NULL)
 *   receives the mean time of one launch.  Synchronises the stream. */
vla_status vla_test_ternary_gemm(const int8_t* q, const float* r, const uint8_t* w_packed, const float* wscale,
                                 int32_t M, int32_t N, int32_t K, int32_t variant, int32_t iters, float* y,
                                 float* us_per_launch, void* stream);

/* Residual finish + adaRMS of the next sublayer (the row kernel that closes
 * every residual branch, scope rows a4 and a7): for every row m of M,
 *   x[m] += alpha * sum_{s < nsplit} part[s][m]      (alpha NULL: no update)
 *   u[m]  = x[m] / sqrt(mean(x[m]^2) + eps) * (1 + gamma) + beta
 * x [M][d] fp32 is updated in place; part [nsplit][M][d] fp32; alpha, gamma,
 * beta [d] fp32; u [M][d] fp32 (u_f32 = 1) or elem (bf16 when elem = 1).
 * d % 4 == 0, d <= 4096. */
vla_status vla_test_adarms(int32_t elem, float* x, const float* part, int32_t nsplit, const float* alpha,
                           const float* gamma, const float* beta, int32_t M, int32_t d, float eps, void* u,
                           int32_t u_f32, void* stream);

/* Time-conditioning precompute of a time-conditioned model (scope row a2):
 * for the HOST schedule t_schedule [n_steps+1], step k uses tau_k:
 * e = sinusoid(tau_k), c = W_t2 SiLU(W_t1 e + b_t1) + b_t2, and
 *   mods [n_steps][L * 3 * n_sub * d] = W_mod SiLU(c) + b_mod   (every layer, stacked)
 *   modf [n_steps][2 d]              = W_fm SiLU(c) + b_fm
 * both fp32 device buffers.  VLA_E_UNSUPPORTED for a regression-head model. */
vla_status vla_test_time_cond(struct vla_model* model, const float* t_schedule, int32_t n_steps, float* mods,
                              float* modf, void* stream);

/* Phase timeline of the model's last persistent vla_denoise call made with
 * VLA_OPT_TRACE = 1: for each of the 8 teams, max_per_team 100 MHz clock
 * values (before and after every barrier, in order; unused entries hold
 * stale data) copied to out [8][max_per_team] (host).  With VLA_OPT_TRACE = 2
 * every workgroup records its first 256 marks: out [256][n], row
 * team * 32 + rank, n = min(max_per_team, 256).  Synchronises the device.
 * Returns the entries copied per row, or -1 if nothing was traced. */
int32_t vla_test_persist_trace(struct vla_model* model, uint64_t* out, int32_t max_per_team);

#ifdef __cplusplus
}
#endif
#endif /* VLA_TEST_H_ */

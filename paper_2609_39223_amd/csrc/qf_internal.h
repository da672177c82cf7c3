// Internal launch interface shared by the C ABI (qf_api.hip) and the kernel files.
// Host-side validation happens in qf_api.hip; the launchers below assume valid arguments.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qf {

// ---- quantizers (qf_quant.hip) ----------------------------------------------------------
// Writes v to p[0..n) with a kernel (no memset nodes, so callers may capture it in a graph).
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s);
// Tensor amax into *amax (accumulate: max(*amax, amax), compared as bits); one dispatch, no
// clearing kernel before it (an empty tensor: a one-element fill unless accumulating).
hipError_t launch_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                       bool accumulate, hipStream_t s);
// g: device scalar holding the tensor amax to use; s_out may be null.  stream_out: write the
// outputs with non-temporal stores (for a call right after an amax pass over the same input
// that fits the last-level cache, whose lines the outputs then do not evict).
hipError_t launch_nvfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, const float* g,
                        float* s_out, uint8_t* codes, uint8_t* scales, uint16_t* xhat,
                        hipStream_t s, bool stream_out = false);
hipError_t launch_mxfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* codes,
                        uint8_t* scales, uint16_t* xhat, hipStream_t s);
hipError_t launch_q4k(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* packed,
                      uint16_t* xhat, hipStream_t s);
// Q4_K with searched sub-block steps (never a larger super-block error than launch_q4k's).
hipError_t launch_q4k_mse(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* packed,
                          uint16_t* xhat, hipStream_t s);

// Batched variants over E equally shaped tensors (expert weights), one tensor scale each.
hipError_t launch_amax_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K,
                               float* amax, bool accumulate, hipStream_t s);
// NVFP4 of tensor z with g[z]: x_hat and, when non-null, S[z], codes and scales of all E tensors
// back to back (tensor z's after tensor z - 1's).
hipError_t launch_nvfp4_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K,
                                const float* g, float* s_out, uint8_t* codes, uint8_t* scales,
                                uint16_t* xhat, hipStream_t s);

// Quantize-dequantize with transposed output: out[k][r] = x_hat[r][k] (bf16, row stride ldo)
// for `batch` tensors spaced xbs / obs elements apart (NVFP4: tensor amax g[z] per tensor).
// R and K multiples of 8, K a multiple of the format block.
hipError_t launch_quant_t(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                          int64_t batch, int64_t xbs, const float* g, uint16_t* out, int64_t ldo,
                          int64_t obs, hipStream_t s);
// Dequantize with transposed output from packed codes: out[k][r] = x_hat[r][k] (bf16, row
// stride ldo) of a [R, K] tensor stored as codes [R][K/2] + scales [R][K/16 | K/32] (NVFP4
// with its tensor decode scale S = g / 2688 at S) or Q4_K blocks [R][K/256][144] (in
// `codes`); bit-identical to launch_quant_t's x_hat of the tensor those codes came from.
// R and K multiples of 8 (Q4K: K of 256).
// batch > 1: that many [R, K] tensors stored back to back (decode scale S[z]), tensor z's
// output obs elements after tensor z - 1's.
hipError_t launch_dequant_t(int fmt, const uint8_t* codes, const uint8_t* scales,
                            const float* S, int64_t R, int64_t K, uint16_t* out, int64_t ldo,
                            hipStream_t s, int64_t batch = 1, int64_t obs = 0);
// Grouped, transposed, 64-padded: rows [off[e], off[e+1]) of x [T, K] (fmt NONE or MXFP4)
// land as columns [64 kstart[e], 64 kstart[e+1]) of out [K, ldo] (x_hat^T), zeros past each
// expert's last row.  kstart from launch_grouped_prep.
hipError_t launch_quant_t_grouped(int fmt, const uint16_t* x, int64_t T, int64_t K,
                                  const int64_t* off, const int* kstart, int64_t E,
                                  uint16_t* out, int64_t ldo, hipStream_t s);

// ---- GEMMs --------------------------------------------------------------------------------
// NT GEMM (qf_gemm_nt.hip): C[m, n] = sum_k A(m, k) B(n, k).  A is [M][K] (k contiguous) or,
// with a_mn, [K][M] (m contiguous); likewise B [N][K] or [K][N] with b_mn.  Row strides and
// K multiples of 8.  With `at` (bf16 C, both operands k-major, M % 8 == 0, M <= ldat <
// kGemmAtMaxLd, ldat a multiple of 4, at 8-byte aligned) the launch also writes A^T [K][M]
// (row stride ldat): from the tiles it stages anyway when N spans at least 8 tile columns,
// else with the transpose kernel; other arguments give hipErrorInvalidValue.
constexpr int64_t kGemmAtMaxLd = (int64_t)1 << 24;
hipError_t launch_gemm_nt(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                          int a_mn, const uint16_t* B, int64_t ldb, int b_mn, void* C,
                          int64_t ldc, int c_f32, float* part, hipStream_t s,
                          uint16_t* at = nullptr, int64_t ldat = 0);
// The same product with B [N, K] given in the fragment-major layout the MFMA operands use
// (launch_frag_pack writes it from a row-major matrix; gemm_frag_bytes(N, K) bytes, rows padded
// to a multiple of 32 with zeros): B's fragments go from memory straight into registers and only
// A is staged in LDS.  A k-major; K a multiple of 64; Bf 16-byte aligned.  Results equal
// launch_gemm_nt's on the row-major B bit for bit.
hipError_t launch_gemm_nt_bf(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                             const uint16_t* Bf, void* C, int64_t ldc, int c_f32, float* part,
                             hipStream_t s, uint16_t* at = nullptr, int64_t ldat = 0);
size_t gemm_frag_bytes(int64_t N, int64_t K);
hipError_t launch_frag_pack(const uint16_t* B, int64_t N, int64_t K, int64_t ld, uint16_t* out,
                            hipStream_t s);
// The forward Y[M, N] = A W_hat^T (bf16 C) with W_hat decoded inside the GEMM from the packed
// weight (bfmt NVFP4 / MXFP4: codes [N][K/2] + scales [N][K/16 | K/32] + NVFP4 tensor decode
// scale S = g / 2688 at S; Q4K: blocks [N][K/256][144] in `codes`).  K a multiple of 64 (Q4K:
// 256); A k-major; codes and scales rows 16-byte aligned (base pointers 16-byte aligned).
hipError_t launch_gemm_nt_packed_b(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                                   int64_t lda, int bfmt, const uint8_t* codes,
                                   const uint8_t* scales, const float* S, uint16_t* C,
                                   int64_t ldc, hipStream_t s);
// Bytes of the FP32 partial buffer `part` an [M, N] FP32-output launch may use (a K-split
// of the last partial round of tiles).  part may be null: no split.
size_t gemm_nt_split_bytes(int64_t M, int64_t N);
// Grouped-K NT (per-expert weight gradient): C + e cstride [M, N] = A[:, k] B[:, k]^T over
// k in [64 kstart[e], 64 kstart[e+1]) of the padded operands A [M][Kpad], B [N][Kpad].
hipError_t launch_grouped_nt_k(int64_t E, int64_t M, int64_t N, int64_t Kpad, const int* kstart,
                                const int* order, const uint16_t* A, int64_t lda,
                                const uint16_t* B, int64_t ldb, float* C, int64_t ldc,
                                int64_t cstride, hipStream_t s);
// Grouped NT: rows [off[e], off[e+1]) of A use B + e * bstride ([N][K], k contiguous, or
// [K][N] with b_mn).  With `at` (k-contiguous B, N spanning at least 8 tile columns, kstart
// from launch_grouped_prep, ldat a multiple of 4 below kGemmAtMaxLd, at 8-byte aligned) the
// launch also writes A^T in the padded layout of the grouped weight gradient: row k, column
// 64 kstart[e] + i holds A[off[e] + i][k], zeros up to 64 kstart[e+1].
hipError_t launch_grouped_nt_rows(int64_t E, int64_t T, int64_t N, int64_t K, const int64_t* off,
                                  const int* tile_start, const uint16_t* A, int64_t lda,
                                  const uint16_t* B, int64_t ldb, int b_mn, int64_t bstride,
                                  uint16_t* C, int64_t ldc, hipStream_t s,
                                  uint16_t* at = nullptr, int64_t ldat = 0,
                                  const int* kstart = nullptr);
// bf16 transpose (qf_transpose.hip): out[c][r] = in[r][c] for `batch` matrices spaced ibs / obs
// elements apart; R and C multiples of 8.
hipError_t launch_transpose_bf16(const uint16_t* in, int64_t R, int64_t C, int64_t ldi,
                                 uint16_t* out, int64_t ldo, int64_t batch, int64_t ibs,
                                 int64_t obs, hipStream_t s);

// Grouped over experts (qf_grouped.hip; rows [off[e], off[e+1]) of the token-major operands belong to
// expert e; the host never reads off).  launch_grouped_prep fills small device arrays:
// tile_start[E+1] (prefix of per-expert 256-row tile counts), order[E] (experts by
// decreasing row count) and, when non-null, kstart[E+1] (prefix of per-expert 64-row counts).
hipError_t launch_grouped_prep(const int64_t* off, int64_t E, int* tile_start, int* order,
                               int* kstart, hipStream_t s);

// ---- LoRA-QAD (qf_lora.hip) ------------------------------------------------------------------
// Low-rank factors of a merged weight W + scale * B A: A FP32 [r, K] (row stride K), B FP32
// [N, r] (row stride r); for `batch` tensors, tensor z uses A + z * a_stride and
// B + z * b_stride (a stride of 0 shares the factor).  A and B 16-byte aligned.
struct LoraOperand {
  const float* A;
  int64_t a_stride;
  const float* B;
  int64_t b_stride;
  int64_t r;
  float scale;
};
// amax of the merged bf16 tensors folded into amax[z] (bit-pattern atomic max; initialize).
hipError_t launch_lora_amax(const LoraOperand& L, const uint16_t* w, int64_t N, int64_t K,
                            int64_t ldw, int64_t batch, int64_t wbs, float* amax, hipStream_t s);
// Quantize-dequantize of the merged tensors (fmt NONE: the merged bf16 tensor itself).  Row
// outputs per tensor z at z * N * (K/2 | K/block | (K/256) * 144 | K); g: NVFP4 amax per tensor.
hipError_t launch_lora_quant(int fmt, const LoraOperand& L, const uint16_t* w, int64_t N,
                             int64_t K, int64_t ldw, int64_t batch, int64_t wbs, const float* g,
                             float* s_out, uint8_t* codes, uint8_t* scales, uint8_t* packed,
                             uint16_t* xhat, hipStream_t s);
// Same with transposed bf16 output out[k][n] (row stride ldo, tensor z at out + z * obs).
hipError_t launch_lora_quant_t(int fmt, const LoraOperand& L, const uint16_t* w, int64_t N,
                               int64_t K, int64_t ldw, int64_t batch, int64_t wbs, const float* g,
                               uint16_t* out, int64_t ldo, int64_t obs, hipStream_t s);
// Grouped (mixture-of-experts) mode of the two kernels below: off [E+1] (device) splits the M
// rows into experts and pre [E+1] (device, launch_group_prefix with the kernel's chunk: 16
// rows for the row-dot, 1024 for the column sum) deals expert-aligned chunks to blocks; off
// null = one group.  pre[e] = sum over experts before e of ceil(rows / q).
hipError_t launch_group_prefix(const int64_t* off, int64_t E, int q, int* pre, hipStream_t s);
// P[m][j] = sum_k X[m][k] F[j][k]: X bf16 [M, K] (ldx a multiple of 8, 16-byte aligned), F FP32
// [r, K] (ldf, multiple of 4, 16-byte aligned; grouped: expert e uses F + e * fstride), P FP32
// [M, ldp] with ldp = r rounded up to 16 (zeros past r).  K a multiple of 8.  Both run on MFMA
// with the FP32 factor split into bf16 hi + lo (within the floating-point tolerance, not the
// FP32 FMA chain's rounding).
hipError_t launch_lora_rowdot(const uint16_t* X, int64_t M, int64_t K, int64_t ldx, const float* F,
                              int64_t ldf, int64_t r, float* P, int64_t ldp, const int64_t* off,
                              const int* pre, int64_t E, int64_t fstride, hipStream_t s);
// out = scale * sum_m Big[m][c] Sm[m][j] as out[c][j] (or out[j][c] when transposed): Big bf16
// [M, C] (16-byte aligned, ldb a multiple of 8, C a multiple of 4), Sm FP32 [M, lds_] as the
// row-dot writes it (lds_ = r
// rounded up to 16, zeros past r, 16-byte aligned); `part` holds lora_colsum_part_bytes(M, C,
// r) bytes (grouped: lora_colsum_grouped_part_bytes) of row-chunk partials, summed in a fixed
// order.  Grouped with per_group: out + e * C * r receives expert e's rows only; grouped
// without: the sum over all rows.
size_t lora_colsum_part_bytes(int64_t M, int64_t C, int64_t r);
size_t lora_colsum_grouped_part_bytes(int64_t T, int64_t E, int64_t C, int64_t r);
hipError_t launch_lora_colsum(const uint16_t* Big, int64_t M, int64_t C, int64_t ldb,
                              const float* Sm, int64_t lds_, int64_t r, float scale,
                              float* part, int transposed, float* out, const int64_t* off,
                              const int* pre, int64_t E, int per_group, hipStream_t s);
// Ft [z][r][N] = F[z]^T for `batch` FP32 [N, r] matrices stored back to back.
hipError_t launch_transpose_f32(const float* F, int64_t N, int64_t r, int64_t batch, float* Ft,
                                hipStream_t s);

// ---- QAD distillation loss (qf_kl.hip) ---------------------------------------------------------
// Per row of bf16 logits [L, V] (V % 8 == 0): row_kl[t], optional loss (mean), grad
// (gscale (p_S - p_T), bf16) and agree (top-1 equality).
hipError_t launch_qad_kl(const uint16_t* zt, int64_t ldt, const uint16_t* zs, int64_t lds_,
                         int64_t L, int64_t V, float gscale, float* row_kl, float* loss,
                         uint16_t* grad, int64_t ldg, int32_t* agree, hipStream_t s);

// ---- export helpers (qf_export.hip) --------------------------------------------------------
// ws2 = *g / 2688 and is = *a / 2688 (either output may be null; a is read only when is is set).
hipError_t launch_export_scalars(const float* g, const float* a, float* ws2, float* is,
                                 hipStream_t s);
// Writes the 64-byte payload header (16 little-endian 32-bit words) to payload.
hipError_t launch_payload_header(void* payload, const uint32_t words[16], hipStream_t s);
}  // namespace qf

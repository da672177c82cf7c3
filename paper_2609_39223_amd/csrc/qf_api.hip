// C ABI of libqf (declared in include/qf.h): host-side validation, workspace layout and the
// launch sequence of each call.  No call allocates device memory or synchronizes; every
// kernel goes on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>

#include "qf.h"
#include "qf_internal.h"

namespace {

thread_local char g_err[512] = "";

qf_status fail(qf_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

qf_status ok() {
  g_err[0] = 0;
  return QF_OK;
}

qf_status dev(hipError_t e, const char* what) {
  if (e == hipSuccess) return QF_OK;
  return fail(QF_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define QF_TRY(expr)                      \
  do {                                    \
    qf_status _st = (expr);               \
    if (_st != QF_OK) return _st;         \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// A 2-D bf16 operand: rows x cols with row stride ld (elements).
qf_status check_mat(const char* name, const void* p, int64_t rows, int64_t cols, int64_t ld,
                    bool required) {
  if (rows < 0 || cols < 0) return fail(QF_ESHAPE, "%s: negative shape", name);
  if (rows == 0 || cols == 0) return QF_OK;
  if (!p) {
    if (required) return fail(QF_EINVAL, "%s: null pointer", name);
    return QF_OK;
  }
  if (ld < cols) return fail(QF_ESHAPE, "%s: row stride %lld < %lld columns", name,
                             (long long)ld, (long long)cols);
  if (!aligned16(p)) return fail(QF_EALIGN, "%s: pointer not 16-byte aligned", name);
  if (ld % 8) return fail(QF_EALIGN, "%s: row stride %lld not a multiple of 8", name,
                          (long long)ld);
  return QF_OK;
}

qf_status check_out(const char* name, const void* p) {
  if (p && !aligned16(p)) return fail(QF_EALIGN, "%s: pointer not 16-byte aligned", name);
  return QF_OK;
}

qf_status check_quant_input(const char* fn, const uint16_t* x, int64_t R, int64_t K,
                            int64_t ldx, int64_t block) {
  if (R < 0 || K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (K % block) return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of the block size %lld",
                             fn, (long long)K, (long long)block);
  return check_mat(fn, x, R, K, ldx, true);
}

inline hipStream_t S(qf_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

constexpr size_t kAlign = 256;
inline size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool fmt_valid(int f) { return f >= QF_FMT_NONE && f <= QF_FMT_Q4K; }

int64_t block_of(int f) {
  switch (f) {
    case QF_FMT_NVFP4: return 16;
    case QF_FMT_MXFP4: return 32;
    case QF_FMT_Q4K: return 256;
    default: return 8;
  }
}

// x_hat-only fake quantization of a [R, K] bf16 tensor into out (row stride K).
// NVFP4: g_given (device) when non-null, else computed into g_scratch.
qf_status fakequant_to(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                       const float* g_given, float* g_scratch, uint16_t* out, hipStream_t s) {
  switch (fmt) {
    case QF_FMT_NVFP4: {
      const float* g = g_given;
      if (!g) {
        QF_TRY(dev(qf::launch_amax(x, R, K, ldx, g_scratch, false, s), "amax"));
        g = g_scratch;
      }
      return dev(qf::launch_nvfp4(x, R, K, ldx, g, nullptr, nullptr, nullptr, out, s), "nvfp4");
    }
    case QF_FMT_MXFP4:
      return dev(qf::launch_mxfp4(x, R, K, ldx, nullptr, nullptr, out, s), "mxfp4");
    case QF_FMT_Q4K:
      return dev(qf::launch_q4k(x, R, K, ldx, nullptr, out, s), "q4k");
    default:
      return fail(QF_EINVAL, "bad format %d", fmt);
  }
}

// A quantized operand in packed form: codes [R][K/2] + block scales [R][K/B] + (NVFP4) the
// tensor decode scale S = g / 2688 in its own 256-byte slot (nS scales, one per tensor, for
// the experts of a grouped layer stored back to back); Q4_K: blocks [R][K/256][144] in
// `codes`.  This is the layer's saved form of W_hat / A_hat (0.5625 bytes per element).
struct Packed {
  uint8_t* codes;
  uint8_t* scales;
  float* S;
};

size_t packed_bytes(int fmt, int64_t R, int64_t K, int64_t nS = 1) {
  const size_t r = R, k = K;
  switch (fmt) {
    case QF_FMT_NVFP4: return up((size_t)nS * 4) + up(r * k / 2) + up(r * k / 16);
    case QF_FMT_MXFP4: return up(r * k / 2) + up(r * k / 32);
    case QF_FMT_Q4K: return up(r * (k / 256) * 144);
    default: return 0;
  }
}

// Carve a packed operand of format fmt out of p (advances p).
Packed carve_packed(int fmt, int64_t R, int64_t K, char*& p, int64_t nS = 1) {
  Packed q{};
  const size_t r = R, k = K;
  if (fmt == QF_FMT_NVFP4) { q.S = reinterpret_cast<float*>(p); p += up((size_t)nS * 4); }
  if (fmt == QF_FMT_NONE) return q;
  q.codes = reinterpret_cast<uint8_t*>(p);
  if (fmt == QF_FMT_Q4K) { p += up(r * (k / 256) * 144); return q; }
  p += up(r * k / 2);
  q.scales = reinterpret_cast<uint8_t*>(p);
  p += up(r * k / (fmt == QF_FMT_NVFP4 ? 16 : 32));
  return q;
}

// The saved operands of one layer call: packed W_hat, then packed A_hat when afmt != NONE.
size_t saved_bytes(const qf_qlinear_desc* d) {
  return packed_bytes(d->wfmt, d->N, d->K) + packed_bytes(d->afmt, d->M, d->K);
}
void saved_layout(const qf_qlinear_desc* d, void* saved, Packed* w, Packed* a) {
  char* p = static_cast<char*>(saved);
  *w = carve_packed(d->wfmt, d->N, d->K, p);
  *a = carve_packed(d->afmt, d->M, d->K, p);
}

// Row stride (elements) of a workspace operand whose rows hold `cols` bf16 values.  Byte strides
// that are multiples of 32 KB put every row of a GEMM tile on the same memory channels and L2
// sets (an NT GEMM over 64 KB strides measured ~5 % slower than over 64 KB + 256 B; 16 KB
// strides showed no difference), so those rows get 128 more elements.
int64_t ws_ld(int64_t cols) { return cols % 16384 == 0 ? cols + 128 : cols; }

// Workspace of one linear layer (256-byte aligned regions):
//   scal   256 B   weight amax scratch
//   wpk    packed W_hat (when wfmt != NONE): the forward's GEMM operand (decoded inside the
//                  GEMM), kept for a QF_FLAG_REUSE_WS backward when no saved buffer is given
//   what   [N, K]  W_hat in bf16 (when wfmt != NONE): the operand of a materializing forward
//                  and of the token-count-not-a-multiple-of-8 backward
//   ahat   [M, K]  A_hat, when afmt != NONE
//   whatt  [K, N]  W_hat^T (or W^T): right operand of dX = dY W_hat in NT form
//   ahatt  [K, M]  A_hat^T (or X^T): right operand of dW = dY^T A_hat in NT form (row stride
//                  ws_ld(M))
//   dyt    [N, M]  dY^T: left operand of dW (row stride ws_ld(M))
//   part   FP32 partial tiles of the dW GEMM's split last round (qf::gemm_nt_split_bytes)
struct LinearWs {
  float* scal;
  Packed wpk;
  uint16_t* what;
  uint16_t* ahat;
  uint16_t* whatt;
  uint16_t* ahatt;
  uint16_t* dyt;
  float* part;
};

size_t linear_ws_bytes(const qf_qlinear_desc* d) {
  const size_t M = d->M, N = d->N, K = d->K;
  size_t b = kAlign;
  if (d->wfmt != QF_FMT_NONE) b += packed_bytes(d->wfmt, d->N, d->K) + up(N * K * 2);
  if (d->afmt != QF_FMT_NONE) b += up(M * K * 2);
  const size_t ldm = (size_t)ws_ld(d->M);
  b += up(K * N * 2) + up(K * ldm * 2) + up(N * ldm * 2);
  b += up(qf::gemm_nt_split_bytes(d->N, d->K));
  return b;
}

LinearWs linear_ws(const qf_qlinear_desc* d, void* ws) {
  const size_t M = d->M, N = d->N, K = d->K;
  char* p = static_cast<char*>(ws);
  LinearWs w{};
  w.scal = reinterpret_cast<float*>(p);
  p += kAlign;
  if (d->wfmt != QF_FMT_NONE) {
    w.wpk = carve_packed(d->wfmt, d->N, d->K, p);
    w.what = reinterpret_cast<uint16_t*>(p); p += up(N * K * 2);
  }
  if (d->afmt != QF_FMT_NONE) { w.ahat = reinterpret_cast<uint16_t*>(p); p += up(M * K * 2); }
  const size_t ldm = (size_t)ws_ld(d->M);
  w.whatt = reinterpret_cast<uint16_t*>(p); p += up(K * N * 2);
  w.ahatt = reinterpret_cast<uint16_t*>(p); p += up(K * ldm * 2);
  w.dyt = reinterpret_cast<uint16_t*>(p); p += up(N * ldm * 2);
  w.part = reinterpret_cast<float*>(p);
  return w;
}

struct Dims {
  int64_t ldx, ldw, ldy;
};

qf_status check_desc(const char* fn, const qf_qlinear_desc* d, Dims* dm) {
  if (!d) return fail(QF_EINVAL, "%s: null descriptor", fn);
  if (d->M < 0 || d->N < 0 || d->K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (!fmt_valid(d->wfmt) || !fmt_valid(d->afmt))
    return fail(QF_EINVAL, "%s: bad format (wfmt=%d afmt=%d)", fn, d->wfmt, d->afmt);
  if (d->afmt == QF_FMT_Q4K)
    return fail(QF_ENOTSUP, "%s: Q4_K is a weight-only format (W4A16)", fn);
  if (d->afmt == QF_FMT_NVFP4 && !d->a_amax)
    return fail(QF_EINVAL, "%s: NVFP4 activations need a_amax (the running amax)", fn);
  const int64_t need = block_of(d->wfmt) > block_of(d->afmt) ? block_of(d->wfmt)
                                                              : block_of(d->afmt);
  if (d->K % need)
    return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of %lld", fn, (long long)d->K,
                (long long)need);
  if (d->N % 8) return fail(QF_ESHAPE, "%s: N=%lld is not a multiple of 8", fn, (long long)d->N);
  dm->ldx = d->ldx ? d->ldx : d->K;
  dm->ldw = d->ldw ? d->ldw : d->K;
  dm->ldy = d->ldy ? d->ldy : d->N;
  return QF_OK;
}

qf_status check_ws(const char* fn, size_t need, void* ws, size_t ws_bytes) {
  if (ws_bytes < need)
    return fail(QF_EINVAL, "%s: workspace %zu bytes < required %zu", fn, ws_bytes, need);
  if (!ws) return fail(QF_EINVAL, "%s: null workspace", fn);
  if ((uintptr_t)ws % kAlign) return fail(QF_EALIGN, "%s: workspace not 256-byte aligned", fn);
  return QF_OK;
}

// Quantize W (and X when afmt != NONE) into the workspace; returns the GEMM operands.
qf_status quantize_operands(const qf_qlinear_desc* d, const Dims& dm, const uint16_t* X,
                            const uint16_t* W, const LinearWs& w, bool do_w, bool do_a,
                            const uint16_t** Wop, int64_t* ldw_op, const uint16_t** Aop,
                            int64_t* lda_op, hipStream_t s) {
  *Wop = W; *ldw_op = dm.ldw;
  *Aop = X; *lda_op = dm.ldx;
  if (d->wfmt != QF_FMT_NONE) {
    if (do_w) QF_TRY(fakequant_to(d->wfmt, W, d->N, d->K, dm.ldw, d->w_amax, w.scal, w.what, s));
    *Wop = w.what; *ldw_op = d->K;
  }
  if (d->afmt != QF_FMT_NONE) {
    if (do_a) QF_TRY(fakequant_to(d->afmt, X, d->M, d->K, dm.ldx, d->a_amax, nullptr, w.ahat, s));
    *Aop = w.ahat; *lda_op = d->K;
  }
  return QF_OK;
}

// Quantize x [R, K] into its packed form pk (codes, block scales, NVFP4 decode scale S) and,
// when xhat is non-null, its bf16 x_hat.  NVFP4: g_given (device) when non-null, else the
// tensor amax computed into g_scratch.
qf_status quantize_packed(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                          const float* g_given, float* g_scratch, const Packed& pk,
                          uint16_t* xhat, hipStream_t s) {
  switch (fmt) {
    case QF_FMT_NVFP4: {
      const float* g = g_given;
      if (!g) {
        QF_TRY(dev(qf::launch_amax(x, R, K, ldx, g_scratch, false, s), "amax"));
        g = g_scratch;
      }
      return dev(qf::launch_nvfp4(x, R, K, ldx, g, pk.S, pk.codes, pk.scales, xhat, s), "nvfp4");
    }
    case QF_FMT_MXFP4:
      return dev(qf::launch_mxfp4(x, R, K, ldx, pk.codes, pk.scales, xhat, s), "mxfp4");
    case QF_FMT_Q4K:
      return dev(qf::launch_q4k(x, R, K, ldx, pk.codes, xhat, s), "q4k");
    default:
      return fail(QF_EINVAL, "bad format %d", fmt);
  }
}

// The forward decodes the packed weight inside the GEMM when the caller asks for it
// (QF_FLAG_DECODE_IN_GEMM) and K is a multiple of the GEMM's 64-deep stages; otherwise it
// writes the bf16 W_hat (the packed operand is written either way).
bool fused_forward(const qf_qlinear_desc* d) {
  return d->wfmt != QF_FMT_NONE && (d->flags & QF_FLAG_DECODE_IN_GEMM) != 0 && d->K > 0 &&
         d->K % 64 == 0 && d->N > 0;
}

// Whether a forward with this descriptor leaves A_hat^T [K, ws_ld(M)] in the workspace (for a
// QF_FLAG_REUSE_WS backward): the materialized forward on a token count that is a multiple of
// 8 (the NT backward's case), with at most 32 output tile columns.  Writing A^T costs the
// forward GEMM a few microseconds per round of tiles plus the pieces it writes; measured at 32K
// tokens (same box) it saves 0.18 / 0.03 / 0.01 ms net for the 4096 x 12288, 4096 x 4096 and
// 6144 x 4096 weights (16-24 tile columns) and loses 0.06 ms for the 24576 x 4096 one (96
// columns, 48 rounds), where the backward's transpose (0.12 ms) is the cheaper route.
bool forward_writes_at(const qf_qlinear_desc* d) {
  return (d->flags & QF_FLAG_REUSE_WS) != 0 && !fused_forward(d) && d->M % 8 == 0 &&
         ws_ld(d->M) < qf::kGemmAtMaxLd && (d->N + 255) / 256 <= 32;
}

qf_status linear_forward(const char* fn, const qf_qlinear_desc* d, const Dims& dm,
                         const uint16_t* X, const uint16_t* W, uint16_t* Y, const LinearWs& w,
                         const Packed& pw, const Packed* pa, hipStream_t s) {
  const bool fused = fused_forward(d);
  const uint16_t* Wop = W;
  int64_t ldw_op = dm.ldw;
  if (d->wfmt != QF_FMT_NONE) {
    QF_TRY(quantize_packed(d->wfmt, W, d->N, d->K, dm.ldw, d->w_amax, w.scal, pw,
                           fused ? nullptr : w.what, s));
    Wop = w.what;
    ldw_op = d->K;
  }
  const uint16_t* Aop = X;
  int64_t lda_op = dm.ldx;
  if (d->afmt != QF_FMT_NONE) {
    if (pa) QF_TRY(quantize_packed(d->afmt, X, d->M, d->K, dm.ldx, d->a_amax, nullptr, *pa, w.ahat, s));
    else QF_TRY(fakequant_to(d->afmt, X, d->M, d->K, dm.ldx, d->a_amax, nullptr, w.ahat, s));
    Aop = w.ahat;
    lda_op = d->K;
  }
  if (fused)
    return dev(qf::launch_gemm_nt_packed_b(d->M, d->N, d->K, Aop, lda_op, d->wfmt, pw.codes,
                                           pw.scales, pw.S, Y, dm.ldy, s),
               fn);
  // With the workspace kept for the backward, the GEMM also writes A_hat^T (X^T when the
  // activations are not quantized), the backward dW's right operand, from the A tiles it
  // stages anyway.
  const bool at = forward_writes_at(d);
  return dev(qf::launch_gemm_nt(d->M, d->N, d->K, Aop, lda_op, 0, Wop, ldw_op, 0, Y, dm.ldy, 0,
                                nullptr, s, at ? w.ahatt : nullptr, ws_ld(d->M)),
             fn);
}

qf_status check_saved(const char* fn, const void* saved) {
  if (saved && (uintptr_t)saved % kAlign)
    return fail(QF_EALIGN, "%s: saved buffer not 256-byte aligned", fn);
  return QF_OK;
}

}  // namespace

extern "C" {

int qf_version(void) { return 200; }

const char* qf_last_error(void) { return g_err; }

qf_status qf_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                  int accumulate, qf_stream_t stream) {
  QF_TRY(check_mat("qf_amax: x", x, R, K, ldx, true));
  if (!amax) return fail(QF_EINVAL, "qf_amax: null amax");
  if (accumulate != 0 && accumulate != 1) return fail(QF_EINVAL, "qf_amax: accumulate must be 0/1");
  QF_TRY(dev(qf::launch_amax(x, R, K, ldx, amax, accumulate != 0, S(stream)), "amax"));
  return ok();
}

qf_status qf_fakequant_nvfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                             int amax_mode, float* s_out, uint8_t* codes, uint8_t* scales,
                             uint16_t* xhat, qf_stream_t stream) {
  QF_TRY(check_quant_input("qf_fakequant_nvfp4", x, R, K, ldx, 16));
  if (!amax) return fail(QF_EINVAL, "qf_fakequant_nvfp4: null amax");
  if (amax_mode != QF_AMAX_COMPUTE && amax_mode != QF_AMAX_GIVEN)
    return fail(QF_EINVAL, "qf_fakequant_nvfp4: bad amax_mode %d", amax_mode);
  if (s_out && s_out == amax) return fail(QF_EINVAL, "qf_fakequant_nvfp4: s_out aliases amax");
  QF_TRY(check_out("qf_fakequant_nvfp4: codes", codes));
  QF_TRY(check_out("qf_fakequant_nvfp4: scales", scales));
  QF_TRY(check_out("qf_fakequant_nvfp4: xhat", xhat));
  hipStream_t s = S(stream);
  if (amax_mode == QF_AMAX_COMPUTE) {
    QF_TRY(dev(qf::launch_amax(x, R, K, ldx, amax, false, s), "amax"));
  }
  if (R == 0 || K == 0) {
    if (s_out) QF_TRY(dev(qf::launch_fill_f32(s_out, 1, 0.0f, s), "S"));
    return ok();
  }
  // After this call's own amax pass, a tensor that fits the 256 MB last-level cache is still
  // there: the quantizer then writes with non-temporal stores so its outputs do not evict it,
  // and its read of x is served from the cache.  A tensor read from HBM anyway keeps plain
  // stores, which are faster there.
  const bool stream_out = amax_mode == QF_AMAX_COMPUTE && R * K * 2 <= (int64_t(160) << 20);
  QF_TRY(dev(qf::launch_nvfp4(x, R, K, ldx, amax, s_out, codes, scales, xhat, s, stream_out),
             "nvfp4"));
  return ok();
}

qf_status qf_fakequant_mxfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, uint16_t* xhat,
                             qf_stream_t stream) {
  QF_TRY(check_quant_input("qf_fakequant_mxfp4", x, R, K, ldx, 32));
  QF_TRY(check_out("qf_fakequant_mxfp4: codes", codes));
  QF_TRY(check_out("qf_fakequant_mxfp4: scales", scales));
  QF_TRY(check_out("qf_fakequant_mxfp4: xhat", xhat));
  QF_TRY(dev(qf::launch_mxfp4(x, R, K, ldx, codes, scales, xhat, S(stream)), "mxfp4"));
  return ok();
}

qf_status qf_fakequant_q4k(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                           uint8_t* packed, uint16_t* xhat, qf_stream_t stream) {
  QF_TRY(check_quant_input("qf_fakequant_q4k", x, R, K, ldx, 256));
  QF_TRY(check_out("qf_fakequant_q4k: packed", packed));
  QF_TRY(check_out("qf_fakequant_q4k: xhat", xhat));
  QF_TRY(dev(qf::launch_q4k(x, R, K, ldx, packed, xhat, S(stream)), "q4k"));
  return ok();
}

qf_status qf_fakequant_q4k_mse(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                               uint8_t* packed, uint16_t* xhat, qf_stream_t stream) {
  QF_TRY(check_quant_input("qf_fakequant_q4k_mse", x, R, K, ldx, 256));
  QF_TRY(check_out("qf_fakequant_q4k_mse: packed", packed));
  QF_TRY(check_out("qf_fakequant_q4k_mse: xhat", xhat));
  QF_TRY(dev(qf::launch_q4k_mse(x, R, K, ldx, packed, xhat, S(stream)), "q4k mse"));
  return ok();
}

qf_status qf_fakequant_transposed(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                                  const float* amax, uint16_t* out, int64_t ldo,
                                  qf_stream_t stream) {
  const char* fn = "qf_fakequant_transposed";
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4 && fmt != QF_FMT_Q4K)
    return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  QF_TRY(check_quant_input(fn, x, R, K, ldx, block_of(fmt)));
  if (R % 8) return fail(QF_ESHAPE, "%s: R=%lld is not a multiple of 8", fn, (long long)R);
  if (R == 0 || K == 0) return ok();
  if (fmt == QF_FMT_NVFP4 && !amax) return fail(QF_EINVAL, "%s: NVFP4 needs amax", fn);
  if (!out) return fail(QF_EINVAL, "%s: null output", fn);
  QF_TRY(check_mat("qf_fakequant_transposed: out", out, K, R, ldo, true));
  QF_TRY(dev(qf::launch_quant_t(fmt, x, R, K, ldx, 1, 0, amax, out, ldo, 0, S(stream)),
             "quantize (transposed)"));
  return ok();
}

qf_status qf_workspace_size(const qf_qlinear_desc* d, size_t* bytes) {
  Dims dm;
  QF_TRY(check_desc("qf_workspace_size", d, &dm));
  if (!bytes) return fail(QF_EINVAL, "qf_workspace_size: null output");
  *bytes = linear_ws_bytes(d);
  return ok();
}

qf_status qf_saved_size(const qf_qlinear_desc* d, size_t* bytes) {
  Dims dm;
  QF_TRY(check_desc("qf_saved_size", d, &dm));
  if (!bytes) return fail(QF_EINVAL, "qf_saved_size: null output");
  *bytes = saved_bytes(d);
  return ok();
}

qf_status qf_qlinear_fwd(const qf_qlinear_desc* d, const uint16_t* X, const uint16_t* W,
                         uint16_t* Y, void* saved, void* ws, size_t ws_bytes,
                         qf_stream_t stream) {
  Dims dm;
  QF_TRY(check_desc("qf_qlinear_fwd", d, &dm));
  QF_TRY(check_mat("qf_qlinear_fwd: X", X, d->M, d->K, dm.ldx, true));
  QF_TRY(check_mat("qf_qlinear_fwd: W", W, d->N, d->K, dm.ldw, true));
  QF_TRY(check_mat("qf_qlinear_fwd: Y", Y, d->M, d->N, dm.ldy, true));
  QF_TRY(check_saved("qf_qlinear_fwd", saved));
  QF_TRY(check_ws("qf_qlinear_fwd", linear_ws_bytes(d), ws, ws_bytes));
  LinearWs w = linear_ws(d, ws);
  Packed pw = w.wpk, pa{};
  if (saved) saved_layout(d, saved, &pw, &pa);
  QF_TRY(linear_forward("forward gemm", d, dm, X, W, Y, w, pw, saved ? &pa : nullptr,
                        S(stream)));
  return ok();
}

}  // extern "C"

// ---------------------------------------------------------------- allocation-free forward
// The forward's quantized operands (W_hat, A_hat and the amax scalar) in a file-scope device
// array instead of a caller workspace.  Each device the library runs on holds its own copy at
// its own address, for the life of the process.  Host code never passes `scratch` itself (in
// host code that name is a stand-in, not a device address): it passes the address that
// hipGetSymbolAddress returns for the current device, looked up once per device.
namespace {

static __device__ __align__(256) char scratch[QF_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

qf_status scratch_of_current_device(void** out) {
  int dev_id = 0;
  QF_TRY(dev(hipGetDevice(&dev_id), "hipGetDevice"));
  if (dev_id < 0 || dev_id >= kMaxDevices)
    return fail(QF_ENOTSUP, "device %d beyond the %d the library tracks", dev_id, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev_id]) {
    void* p = nullptr;
    QF_TRY(dev(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
    if (!p || (uintptr_t)p % kAlign) return fail(QF_EDEVICE, "scratch address not usable");
    g_scratch_ptr[dev_id] = p;
  }
  *out = g_scratch_ptr[dev_id];
  return QF_OK;
}

// Bytes of the forward's operands: the scalar slot, W_hat [N, K] and A_hat [M, K] (bf16).
size_t fwd_operand_bytes(const qf_qlinear_desc* d) {
  const size_t M = d->M, N = d->N, K = d->K;
  size_t b = kAlign;
  if (d->wfmt != QF_FMT_NONE) b += up(N * K * 2);
  if (d->afmt != QF_FMT_NONE) b += up(M * K * 2);
  return b;
}

}  // namespace

extern "C" {

qf_status qf_qlinear_fwd_noalloc(const qf_qlinear_desc* d, const uint16_t* X, const uint16_t* W,
                                 uint16_t* Y, qf_stream_t stream) {
  Dims dm;
  QF_TRY(check_desc("qf_qlinear_fwd_noalloc", d, &dm));
  QF_TRY(check_mat("qf_qlinear_fwd_noalloc: X", X, d->M, d->K, dm.ldx, true));
  QF_TRY(check_mat("qf_qlinear_fwd_noalloc: W", W, d->N, d->K, dm.ldw, true));
  QF_TRY(check_mat("qf_qlinear_fwd_noalloc: Y", Y, d->M, d->N, dm.ldy, true));
  const size_t need = fwd_operand_bytes(d);
  if (need > (size_t)QF_NOALLOC_SCRATCH_BYTES)
    return fail(QF_ESHAPE, "qf_qlinear_fwd_noalloc: the quantized operands need %zu bytes, "
                "beyond the %zu-byte static scratch", need, (size_t)QF_NOALLOC_SCRATCH_BYTES);
  void* base = nullptr;
  QF_TRY(scratch_of_current_device(&base));
  char* p = static_cast<char*>(base);
  LinearWs w{};
  w.scal = reinterpret_cast<float*>(p);   // the amax slot is rewritten per call
  p += kAlign;
  if (d->wfmt != QF_FMT_NONE) { w.what = reinterpret_cast<uint16_t*>(p); p += up((size_t)d->N * d->K * 2); }
  if (d->afmt != QF_FMT_NONE) w.ahat = reinterpret_cast<uint16_t*>(p);
  hipStream_t s = S(stream);
  const uint16_t *Wop, *Aop;
  int64_t ldw_op, lda_op;
  QF_TRY(quantize_operands(d, dm, X, W, w, true, true, &Wop, &ldw_op, &Aop, &lda_op, s));
  QF_TRY(dev(qf::launch_gemm_nt(d->M, d->N, d->K, Aop, lda_op, 0, Wop, ldw_op, 0, Y, dm.ldy, 0,
                                nullptr, s),
             "forward gemm"));
  return ok();
}

qf_status qf_qlinear_bwd_ste(const qf_qlinear_desc* d, const uint16_t* dY, const uint16_t* X,
                             const uint16_t* W, const void* saved, uint16_t* dX, float* dW,
                             void* ws, size_t ws_bytes, qf_stream_t stream) {
  Dims dm;
  QF_TRY(check_desc("qf_qlinear_bwd_ste", d, &dm));
  QF_TRY(check_mat("qf_qlinear_bwd_ste: dY", dY, d->M, d->N, dm.ldy, true));
  QF_TRY(check_mat("qf_qlinear_bwd_ste: X", X, d->M, d->K, dm.ldx, dW != nullptr));
  QF_TRY(check_mat("qf_qlinear_bwd_ste: W", W, d->N, d->K, dm.ldw, dX != nullptr));
  QF_TRY(check_mat("qf_qlinear_bwd_ste: dX", dX, d->M, d->K, dm.ldx, false));
  QF_TRY(check_out("qf_qlinear_bwd_ste: dW", dW));
  QF_TRY(check_saved("qf_qlinear_bwd_ste", saved));
  QF_TRY(check_ws("qf_qlinear_bwd_ste", linear_ws_bytes(d), ws, ws_bytes));
  hipStream_t s = S(stream);
  LinearWs w = linear_ws(d, ws);
  const bool reuse = (d->flags & QF_FLAG_REUSE_WS) != 0;
  // Packed W_hat / A_hat of the forward: from `saved`, else (QF_FLAG_REUSE_WS) W_hat from the
  // workspace's packed region; otherwise the operands are quantized again (identical bits).
  Packed sw{}, sa{};
  if (saved) saved_layout(d, const_cast<void*>(saved), &sw, &sa);
  const Packed* src_w = saved ? &sw : (reuse ? &w.wpk : nullptr);
  if (d->M % 8 == 0) {
    // NT form: transposed operands through the workspace.  W_hat^T comes from the packed
    // operand (transposing dequantizer) or straight from the transposing quantizer (one pass
    // over W).  dY^T (left operand of dW) is written by the dX GEMM from the dY tiles it stages
    // anyway when both gradients are asked for; otherwise by the transpose kernel.
    const int64_t ldm = ws_ld(d->M);
    const bool dyt_by_dx = dX != nullptr && dW != nullptr && ldm < qf::kGemmAtMaxLd;
    if (dX) {  // dX[M, K] = dY[M, N] (W_hat^T)[K, N]^T
      if (d->wfmt != QF_FMT_NONE) {
        if (src_w) {
          QF_TRY(dev(qf::launch_dequant_t(d->wfmt, src_w->codes, src_w->scales, src_w->S, d->N,
                                          d->K, w.whatt, d->N, s), "dequantize W (transposed)"));
        } else {
          const float* g = d->w_amax;
          if (d->wfmt == QF_FMT_NVFP4 && !g) {
            QF_TRY(dev(qf::launch_amax(W, d->N, d->K, dm.ldw, w.scal, false, s), "amax"));
            g = w.scal;
          }
          QF_TRY(dev(qf::launch_quant_t(d->wfmt, W, d->N, d->K, dm.ldw, 1, 0, g, w.whatt, d->N, 0,
                                        s), "quantize W (transposed)"));
        }
      } else {
        QF_TRY(dev(qf::launch_transpose_bf16(W, d->N, d->K, dm.ldw, w.whatt, d->N, 1, 0, 0, s),
                   "transpose W"));
      }
      QF_TRY(dev(qf::launch_gemm_nt(d->M, d->K, d->N, dY, dm.ldy, 0, w.whatt, d->N, 0, dX,
                                    dm.ldx, 0, nullptr, s, dyt_by_dx ? w.dyt : nullptr, ldm),
                 "dX gemm"));
    }
    if (dW) {  // dW[N, K] = (dY^T)[N, M] (A_hat^T)[K, M]^T
      if (!dyt_by_dx)
        QF_TRY(dev(qf::launch_transpose_bf16(dY, d->M, d->N, dm.ldy, w.dyt, ldm, 1, 0, 0, s),
                   "transpose dY"));
      if (forward_writes_at(d)) {
        // A_hat^T is in the workspace already: the forward's GEMM wrote it
      } else if (d->afmt != QF_FMT_NONE && saved) {
        QF_TRY(dev(qf::launch_dequant_t(d->afmt, sa.codes, sa.scales, sa.S, d->M, d->K, w.ahatt,
                                        ldm, s), "dequantize X (transposed)"));
      } else if (d->afmt != QF_FMT_NONE && !reuse) {
        QF_TRY(dev(qf::launch_quant_t(d->afmt, X, d->M, d->K, dm.ldx, 1, 0, d->a_amax, w.ahatt,
                                      ldm, 0, s), "quantize X (transposed)"));
      } else {
        const uint16_t* src = d->afmt != QF_FMT_NONE ? w.ahat : X;
        const int64_t ld = d->afmt != QF_FMT_NONE ? d->K : dm.ldx;
        QF_TRY(dev(qf::launch_transpose_bf16(src, d->M, d->K, ld, w.ahatt, ldm, 1, 0, 0, s),
                   "transpose A_hat"));
      }
      QF_TRY(dev(qf::launch_gemm_nt(d->N, d->K, d->M, w.dyt, ldm, 0, w.ahatt, ldm, 0, dW, d->K,
                                    1, w.part, s),
                 "dW gemm"));
    }
  } else {
    // Token count not a multiple of 8 (no 16-byte transposed rows): the NT kernel reads
    // W_hat [N, K], dY [M, N] and A_hat [M, K] in place as operands stored [K'][*], through
    // transposing LDS reads (slower than the transposed operands, correct for any M).  W_hat is
    // quantized again into the workspace (the forward may have left only its packed form);
    // A_hat is the forward's with QF_FLAG_REUSE_WS.
    const uint16_t *Wop, *Aop;
    int64_t ldw_op, lda_op;
    QF_TRY(quantize_operands(d, dm, X, W, w, dX != nullptr, !reuse && dW != nullptr,
                             &Wop, &ldw_op, &Aop, &lda_op, s));
    if (dX)  // dX[M, K] = dY[M, N] W_hat[N, K]
      QF_TRY(dev(qf::launch_gemm_nt(d->M, d->K, d->N, dY, dm.ldy, 0, Wop, ldw_op, 1, dX, dm.ldx,
                                    0, nullptr, s),
                 "dX gemm"));
    if (dW)  // dW[N, K] = dY[M, N]^T A_hat[M, K]
      QF_TRY(dev(qf::launch_gemm_nt(d->N, d->K, d->M, dY, dm.ldy, 1, Aop, lda_op, 1, dW, d->K, 1,
                                    w.part, s),
                 "dW gemm"));
  }
  return ok();
}

// ------------------------------------------------------------------------------ grouped
namespace {

struct GroupedWs {
  int* tile_start;  // [E+1]
  int* order;       // [E]
  float* wamax;     // [E]
  uint16_t* what;   // [E, N, K]
  uint16_t* ahat;   // [T, K]
  uint16_t* whatt;  // [E, K, N]: per-expert W_hat^T, right operand of dX in NT form
  int* kstart;      // [E+1]: expert e's tokens at padded columns [64 kstart[e], 64 kstart[e+1])
  uint16_t* dyt;    // [N, Tpad] (row stride ws_ld(Tpad)): dY^T, each expert's tokens padded
                    // to a multiple of 64
  uint16_t* at;     // [K, Tpad] (same row stride): A_hat^T, same padding (dW operands, NT form)
};

// Padded token count: each expert's rows rounded up to a multiple of 64.
int64_t grouped_tpad(const qf_grouped_desc* d) { return (d->T + 63 * d->E + 63) / 64 * 64; }

size_t grouped_ws_bytes(const qf_grouped_desc* d) {
  size_t b = up((size_t)(d->E + 1) * 4) + up((size_t)d->E * 4) + up((size_t)d->E * 4);
  if (d->wfmt != QF_FMT_NONE) b += up((size_t)d->E * d->N * d->K * 2);
  if (d->afmt != QF_FMT_NONE) b += up((size_t)d->T * d->K * 2);
  b += up((size_t)d->E * d->N * d->K * 2);
  b += up((size_t)(d->E + 1) * 4);
  const size_t ldt = (size_t)ws_ld(grouped_tpad(d));
  b += up((size_t)d->N * ldt * 2) + up((size_t)d->K * ldt * 2);
  return b;
}

GroupedWs grouped_ws(const qf_grouped_desc* d, void* ws) {
  char* p = static_cast<char*>(ws);
  GroupedWs g{};
  g.tile_start = reinterpret_cast<int*>(p); p += up((size_t)(d->E + 1) * 4);
  g.order = reinterpret_cast<int*>(p); p += up((size_t)d->E * 4);
  g.wamax = reinterpret_cast<float*>(p); p += up((size_t)d->E * 4);
  if (d->wfmt != QF_FMT_NONE) { g.what = reinterpret_cast<uint16_t*>(p); p += up((size_t)d->E * d->N * d->K * 2); }
  if (d->afmt != QF_FMT_NONE) { g.ahat = reinterpret_cast<uint16_t*>(p); p += up((size_t)d->T * d->K * 2); }
  g.whatt = reinterpret_cast<uint16_t*>(p); p += up((size_t)d->E * d->N * d->K * 2);
  g.kstart = reinterpret_cast<int*>(p); p += up((size_t)(d->E + 1) * 4);
  g.dyt = reinterpret_cast<uint16_t*>(p); p += up((size_t)d->N * ws_ld(grouped_tpad(d)) * 2);
  g.at = reinterpret_cast<uint16_t*>(p);
  return g;
}

// The grouped layer's saved operand: the experts' packed W_hat back to back, one tensor
// decode scale per expert (NVFP4); nothing for an unquantized weight.
size_t grouped_saved_bytes(const qf_grouped_desc* d) {
  return packed_bytes(d->wfmt, d->E * d->N, d->K, d->E);
}
Packed grouped_saved_layout(const qf_grouped_desc* d, void* saved) {
  char* p = static_cast<char*>(saved);
  return carve_packed(d->wfmt, d->E * d->N, d->K, p, d->E);
}

qf_status check_grouped(const char* fn, const qf_grouped_desc* d, const int64_t* off) {
  if (!d) return fail(QF_EINVAL, "%s: null descriptor", fn);
  if (d->E < 0 || d->T < 0 || d->N < 0 || d->K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (d->E > 1024) return fail(QF_ENOTSUP, "%s: more than 1024 experts", fn);
  if (!fmt_valid(d->wfmt) || !fmt_valid(d->afmt)) return fail(QF_EINVAL, "%s: bad format", fn);
  if (d->afmt != QF_FMT_NONE && d->afmt != QF_FMT_MXFP4)
    return fail(QF_ENOTSUP, "%s: grouped activations support NONE or MXFP4", fn);
  const int64_t need = block_of(d->wfmt) > block_of(d->afmt) ? block_of(d->wfmt) : block_of(d->afmt);
  if (d->K % need) return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of %lld", fn, (long long)d->K, (long long)need);
  if (d->N % 8) return fail(QF_ESHAPE, "%s: N not a multiple of 8", fn);
  if (d->E > 0 && !off) return fail(QF_EINVAL, "%s: null group_offsets", fn);
  return QF_OK;
}

// W_hat (and, with pk, the experts' packed W_hat in the same launch) and A_hat.
qf_status grouped_quantize(const qf_grouped_desc* d, const uint16_t* X, const uint16_t* W,
                           const GroupedWs& g, bool do_w, bool do_a, const uint16_t** Wop,
                           const uint16_t** Aop, hipStream_t s, const Packed* pk = nullptr) {
  *Wop = W;
  *Aop = X;
  const int64_t R = d->N, K = d->K;
  const Packed q = pk ? *pk : Packed{};
  if (d->wfmt != QF_FMT_NONE) {
    if (do_w) {
      switch (d->wfmt) {
        case QF_FMT_NVFP4: {
          const float* gp = d->w_amax;
          if (!gp) {
            QF_TRY(dev(qf::launch_amax_batched(W, d->E, R, K, g.wamax, false, s), "amax"));
            gp = g.wamax;
          }
          QF_TRY(dev(qf::launch_nvfp4_batched(W, d->E, R, K, gp, q.S, q.codes, q.scales, g.what,
                                              s),
                     "nvfp4"));
          break;
        }
        case QF_FMT_MXFP4:
          QF_TRY(dev(qf::launch_mxfp4(W, d->E * R, K, K, q.codes, q.scales, g.what, s), "mxfp4"));
          break;
        case QF_FMT_Q4K:
          QF_TRY(dev(qf::launch_q4k(W, d->E * R, K, K, q.codes, g.what, s), "q4k"));
          break;
      }
    }
    *Wop = g.what;
  }
  if (d->afmt == QF_FMT_MXFP4) {
    if (do_a) QF_TRY(dev(qf::launch_mxfp4(X, d->T, K, K, nullptr, nullptr, g.ahat, s), "mxfp4"));
    *Aop = g.ahat;
  }
  return QF_OK;
}

}  // namespace

qf_status qf_grouped_workspace_size(const qf_grouped_desc* d, size_t* bytes) {
  QF_TRY(check_grouped("qf_grouped_workspace_size", d, (const int64_t*)1));
  if (!bytes) return fail(QF_EINVAL, "qf_grouped_workspace_size: null output");
  *bytes = grouped_ws_bytes(d);
  return ok();
}

qf_status qf_grouped_saved_size(const qf_grouped_desc* d, size_t* bytes) {
  QF_TRY(check_grouped("qf_grouped_saved_size", d, (const int64_t*)1));
  if (!bytes) return fail(QF_EINVAL, "qf_grouped_saved_size: null output");
  *bytes = grouped_saved_bytes(d);
  return ok();
}

qf_status qf_qlinear_grouped_fwd(const qf_grouped_desc* d, const int64_t* group_offsets,
                                 const uint16_t* X, const uint16_t* W, uint16_t* Y, void* saved,
                                 void* ws, size_t ws_bytes, qf_stream_t stream) {
  QF_TRY(check_grouped("qf_qlinear_grouped_fwd", d, group_offsets));
  QF_TRY(check_mat("qf_qlinear_grouped_fwd: X", X, d->T, d->K, d->K, true));
  QF_TRY(check_mat("qf_qlinear_grouped_fwd: W", W, d->E * d->N, d->K, d->K, true));
  QF_TRY(check_mat("qf_qlinear_grouped_fwd: Y", Y, d->T, d->N, d->N, true));
  QF_TRY(check_saved("qf_qlinear_grouped_fwd", saved));
  QF_TRY(check_ws("qf_qlinear_grouped_fwd", grouped_ws_bytes(d), ws, ws_bytes));
  if (d->E == 0) return ok();
  hipStream_t s = S(stream);
  GroupedWs g = grouped_ws(d, ws);
  const uint16_t *Wop, *Aop;
  const Packed pk = saved ? grouped_saved_layout(d, saved) : Packed{};
  QF_TRY(grouped_quantize(d, X, W, g, true, true, &Wop, &Aop, s, saved ? &pk : nullptr));
  QF_TRY(dev(qf::launch_grouped_prep(group_offsets, d->E, g.tile_start, g.order, g.kstart, s),
             "prep"));
  QF_TRY(dev(qf::launch_grouped_nt_rows(d->E, d->T, d->N, d->K, group_offsets, g.tile_start, Aop,
                                        d->K, Wop, d->K, 0, d->N * d->K, Y, d->N, s),
             "grouped forward"));
  return ok();
}

qf_status qf_qlinear_grouped_bwd_ste(const qf_grouped_desc* d, const int64_t* group_offsets,
                                     const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                                     const void* saved, uint16_t* dX, float* dW, void* ws,
                                     size_t ws_bytes, qf_stream_t stream) {
  QF_TRY(check_grouped("qf_qlinear_grouped_bwd_ste", d, group_offsets));
  QF_TRY(check_mat("qf_qlinear_grouped_bwd_ste: dY", dY, d->T, d->N, d->N, true));
  QF_TRY(check_mat("qf_qlinear_grouped_bwd_ste: X", X, d->T, d->K, d->K, dW != nullptr));
  QF_TRY(check_mat("qf_qlinear_grouped_bwd_ste: W", W, d->E * d->N, d->K, d->K, dX != nullptr));
  QF_TRY(check_mat("qf_qlinear_grouped_bwd_ste: dX", dX, d->T, d->K, d->K, false));
  QF_TRY(check_out("qf_qlinear_grouped_bwd_ste: dW", dW));
  QF_TRY(check_saved("qf_qlinear_grouped_bwd_ste", saved));
  QF_TRY(check_ws("qf_qlinear_grouped_bwd_ste", grouped_ws_bytes(d), ws, ws_bytes));
  if (d->E == 0) return ok();
  hipStream_t s = S(stream);
  GroupedWs g = grouped_ws(d, ws);
  const bool reuse = (d->flags & QF_FLAG_REUSE_WS) != 0;
  // The experts' W_hat^T: dequantized from the saved packed experts, or straight from the
  // transposing quantizer, or (QF_FLAG_REUSE_WS) transposed from the workspace's W_hat.
  const bool from_saved = dX && d->wfmt != QF_FMT_NONE && saved != nullptr;
  const bool fuse_w = dX && d->wfmt != QF_FMT_NONE && !reuse && !from_saved;
  const uint16_t *Wop, *Aop;
  QF_TRY(grouped_quantize(d, X, W, g, !reuse && dX && !fuse_w && !from_saved, false, &Wop,
                          &Aop, s));
  QF_TRY(dev(qf::launch_grouped_prep(group_offsets, d->E, g.tile_start, g.order, g.kstart, s),
             "prep"));
  // dY^T in the padded layout of dW is written by the dX launch from the dY tiles it stages
  // when both gradients are asked for and dX spans at least 8 tile columns (K >= 1793);
  // otherwise by the grouped transposer
  const int64_t tp = grouped_tpad(d), ldt = ws_ld(tp);
  const bool dyt_by_dx = dX != nullptr && dW != nullptr && (d->K + 255) / 256 >= 8 &&
                         ldt < qf::kGemmAtMaxLd;
  if (dX) {
    if (from_saved) {
      const Packed pk = grouped_saved_layout(d, const_cast<void*>(saved));
      QF_TRY(dev(qf::launch_dequant_t(d->wfmt, pk.codes, pk.scales, pk.S, d->N, d->K, g.whatt,
                                      d->N, s, d->E, d->N * d->K),
                 "dequantize saved expert W (transposed)"));
    } else if (fuse_w) {
      const float* gp = d->w_amax;
      if (d->wfmt == QF_FMT_NVFP4 && !gp) {
        QF_TRY(dev(qf::launch_amax_batched(W, d->E, d->N, d->K, g.wamax, false, s), "amax"));
        gp = g.wamax;
      }
      QF_TRY(dev(qf::launch_quant_t(d->wfmt, W, d->N, d->K, d->K, d->E, d->N * d->K, gp, g.whatt,
                                    d->N, d->N * d->K, s),
                 "quantize expert W (transposed)"));
    } else {
      QF_TRY(dev(qf::launch_transpose_bf16(Wop, d->N, d->K, d->K, g.whatt, d->N, d->E,
                                           d->N * d->K, d->N * d->K, s),
                 "transpose expert W_hat"));
    }
    QF_TRY(dev(qf::launch_grouped_nt_rows(d->E, d->T, d->K, d->N, group_offsets, g.tile_start, dY,
                                          d->N, g.whatt, d->N, 0, d->N * d->K, dX, d->K, s,
                                          dyt_by_dx ? g.dyt : nullptr, ldt, g.kstart),
               "grouped dX"));
  }
  if (dW) {
    // dW_e = dY_e^T A_hat_e as one NT launch over padded, transposed token columns: expert e
    // contracts over its own 64-aligned column range (zeros past its last token).
    if (!dyt_by_dx)
      QF_TRY(dev(qf::launch_quant_t_grouped(QF_FMT_NONE, dY, d->T, d->N, group_offsets, g.kstart,
                                            d->E, g.dyt, ldt, s),
                 "transpose dY (grouped)"));
    const bool saved = d->afmt != QF_FMT_NONE && reuse;
    QF_TRY(dev(qf::launch_quant_t_grouped(saved ? QF_FMT_NONE : d->afmt, saved ? g.ahat : X, d->T,
                                          d->K, group_offsets, g.kstart, d->E, g.at, ldt, s),
               "quantize A (grouped, transposed)"));
    QF_TRY(dev(qf::launch_grouped_nt_k(d->E, d->N, d->K, tp, g.kstart, g.order, g.dyt, ldt, g.at,
                                       ldt, dW, d->K, d->N * d->K, s),
               "grouped dW"));
  }
  return ok();
}

qf_status qf_gemm_bf16_ws(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                          int a_kmajor, const uint16_t* B, int64_t ldb, int b_kmajor, void* C,
                          int64_t ldc, int c_f32, void* ws, size_t ws_bytes, qf_stream_t stream) {
  if (M < 0 || N < 0 || K < 0) return fail(QF_ESHAPE, "qf_gemm_bf16: negative shape");
  if ((a_kmajor | b_kmajor | c_f32) & ~1) return fail(QF_EINVAL, "qf_gemm_bf16: flags must be 0/1");
  if (a_kmajor ? false : (M % 8 != 0)) return fail(QF_ESHAPE, "qf_gemm_bf16: M must be a multiple of 8 for [K][M] A");
  if (b_kmajor ? false : (N % 8 != 0)) return fail(QF_ESHAPE, "qf_gemm_bf16: N must be a multiple of 8 for [K][N] B");
  if ((a_kmajor || b_kmajor) && K % 8) return fail(QF_ESHAPE, "qf_gemm_bf16: K must be a multiple of 8");
  QF_TRY(a_kmajor ? check_mat("qf_gemm_bf16: A", A, M, K, lda, true)
                  : check_mat("qf_gemm_bf16: A", A, K, M, lda, true));
  QF_TRY(b_kmajor ? check_mat("qf_gemm_bf16: B", B, N, K, ldb, true)
                  : check_mat("qf_gemm_bf16: B", B, K, N, ldb, true));
  if (M > 0 && N > 0) {
    if (!C) return fail(QF_EINVAL, "qf_gemm_bf16: null C");
    if (ldc < N) return fail(QF_ESHAPE, "qf_gemm_bf16: ldc < N");
    if (!aligned16(C)) return fail(QF_EALIGN, "qf_gemm_bf16: C not 16-byte aligned");
  }
  float* part = nullptr;
  if (ws != nullptr && c_f32) {
    if ((uintptr_t)ws % kAlign) return fail(QF_EALIGN, "qf_gemm_bf16_ws: workspace not 256-byte aligned");
    if (ws_bytes < qf::gemm_nt_split_bytes(M, N))
      return fail(QF_EINVAL, "qf_gemm_bf16_ws: workspace %zu bytes < required %zu", ws_bytes,
                  qf::gemm_nt_split_bytes(M, N));
    part = static_cast<float*>(ws);
  }
  QF_TRY(dev(qf::launch_gemm_nt(M, N, K, A, lda, !a_kmajor, B, ldb, !b_kmajor, C, ldc, c_f32,
                                part, S(stream)),
             "gemm"));
  return ok();
}

qf_status qf_gemm_bf16_at(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                          const uint16_t* B, int64_t ldb, uint16_t* C, int64_t ldc, uint16_t* at,
                          int64_t ldat, qf_stream_t stream) {
  if (M < 0 || N < 0 || K < 0) return fail(QF_ESHAPE, "qf_gemm_bf16_at: negative shape");
  if (M % 8 || K % 8) return fail(QF_ESHAPE, "qf_gemm_bf16_at: M and K must be multiples of 8");
  QF_TRY(check_mat("qf_gemm_bf16_at: A", A, M, K, lda, true));
  QF_TRY(check_mat("qf_gemm_bf16_at: B", B, N, K, ldb, true));
  if (M > 0 && N > 0) {
    if (!C) return fail(QF_EINVAL, "qf_gemm_bf16_at: null C");
    if (ldc < N) return fail(QF_ESHAPE, "qf_gemm_bf16_at: ldc < N");
    if (!aligned16(C)) return fail(QF_EALIGN, "qf_gemm_bf16_at: C not 16-byte aligned");
  }
  if (M > 0 && K > 0) {
    if (!at) return fail(QF_EINVAL, "qf_gemm_bf16_at: null at");
    if (ldat < M || ldat % 4 || ldat >= qf::kGemmAtMaxLd)
      return fail(QF_ESHAPE, "qf_gemm_bf16_at: ldat must be >= M, a multiple of 4 and < 2^24");
    if ((uintptr_t)at % 16) return fail(QF_EALIGN, "qf_gemm_bf16_at: at not 16-byte aligned");
  }
  QF_TRY(dev(qf::launch_gemm_nt(M, N, K, A, lda, 0, B, ldb, 0, C, ldc, 0, nullptr, S(stream),
                                at, ldat),
             "gemm (A^T output)"));
  return ok();
}

qf_status qf_gemm_bf16(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                       int a_kmajor, const uint16_t* B, int64_t ldb, int b_kmajor, void* C,
                       int64_t ldc, int c_f32, qf_stream_t stream) {
  return qf_gemm_bf16_ws(M, N, K, A, lda, a_kmajor, B, ldb, b_kmajor, C, ldc, c_f32, nullptr, 0,
                         stream);
}

qf_status qf_gemm_workspace_size(int64_t M, int64_t N, int c_f32, size_t* bytes) {
  if (!bytes) return fail(QF_EINVAL, "qf_gemm_workspace_size: null output");
  if (M < 0 || N < 0) return fail(QF_ESHAPE, "qf_gemm_workspace_size: negative shape");
  *bytes = c_f32 ? qf::gemm_nt_split_bytes(M, N) : 0;
  return ok();
}

qf_status qf_transpose_bf16(const uint16_t* in, int64_t R, int64_t C, int64_t ldi, uint16_t* out,
                            int64_t ldo, qf_stream_t stream) {
  if (R < 0 || C < 0) return fail(QF_ESHAPE, "qf_transpose_bf16: negative shape");
  if (R % 8 || C % 8) return fail(QF_ESHAPE, "qf_transpose_bf16: R and C must be multiples of 8");
  QF_TRY(check_mat("qf_transpose_bf16: in", in, R, C, ldi, true));
  QF_TRY(check_mat("qf_transpose_bf16: out", out, C, R, ldo, true));
  QF_TRY(dev(qf::launch_transpose_bf16(in, R, C, ldi, out, ldo, 1, 0, 0, S(stream)), "transpose"));
  return ok();
}

// ------------------------------------------------------------------------------- LoRA-QAD
namespace {

constexpr int64_t kMaxRank = 4096;

qf_status check_lora(const char* fn, const qf_lora* L, int64_t N, int64_t K) {
  if (!L) return fail(QF_EINVAL, "%s: null lora", fn);
  if (L->r < 1 || L->r > kMaxRank)
    return fail(QF_ESHAPE, "%s: rank %lld outside [1, %lld]", fn, (long long)L->r,
                (long long)kMaxRank);
  if (N > 0 && K > 0) {
    if (!L->A || !L->B) return fail(QF_EINVAL, "%s: null LoRA factor", fn);
    if (!aligned16(L->A) || !aligned16(L->B))
      return fail(QF_EALIGN, "%s: LoRA factors must be 16-byte aligned", fn);
  }
  return QF_OK;
}

qf::LoraOperand lora_op(const qf_lora* L) {
  return qf::LoraOperand{L->A, 0, L->B, 0, L->r, L->scale};
}

// Workspace of the LoRA layer (256-byte aligned regions):
//   scal  256 B    merged-weight amax scratch
//   what  [N, K]   W_hat of the merged weight (forward operand; kept for a REUSE backward)
//   ahat  [M, K]   A_hat, when afmt != NONE
//   whatt [K, N]   W_hat^T: right operand of dX = dY W_hat in NT form
//   bt    [r, N]   B^T (FP32)
//   u, v  [M, rp]  A_hat A^T and dY B (FP32, rp = r rounded up to 16, zeros past r)
//   part           FP32 row-split partials of the column sums
struct LoraWs {
  float* scal;
  uint16_t* what;
  uint16_t* ahat;
  uint16_t* whatt;
  float* bt;
  float* u;
  float* v;
  float* part;
};

size_t lora_ws_bytes(const qf_qlinear_desc* d, int64_t r) {
  const size_t M = d->M, N = d->N, K = d->K, R = r;
  size_t b = kAlign + up(N * K * 2);
  if (d->afmt != QF_FMT_NONE) b += up(M * K * 2);
  const size_t RP = (R + 15) / 16 * 16;
  b += up(K * N * 2) + up(R * N * 4) + 2 * up(M * RP * 4);
  const size_t p1 = qf::lora_colsum_part_bytes(d->M, d->N, r);
  const size_t p2 = qf::lora_colsum_part_bytes(d->M, d->K, r);
  return b + up(p1 > p2 ? p1 : p2);
}

LoraWs lora_ws(const qf_qlinear_desc* d, int64_t r, void* ws) {
  const size_t M = d->M, N = d->N, K = d->K, R = r, RP = (R + 15) / 16 * 16;
  char* p = static_cast<char*>(ws);
  LoraWs w{};
  w.scal = reinterpret_cast<float*>(p); p += kAlign;
  w.what = reinterpret_cast<uint16_t*>(p); p += up(N * K * 2);
  if (d->afmt != QF_FMT_NONE) { w.ahat = reinterpret_cast<uint16_t*>(p); p += up(M * K * 2); }
  w.whatt = reinterpret_cast<uint16_t*>(p); p += up(K * N * 2);
  w.bt = reinterpret_cast<float*>(p); p += up(R * N * 4);
  w.u = reinterpret_cast<float*>(p); p += up(M * RP * 4);
  w.v = reinterpret_cast<float*>(p); p += up(M * RP * 4);
  w.part = reinterpret_cast<float*>(p);
  return w;
}

// NVFP4 tensor amax of the merged weight: the caller's tied-group value, else computed.
qf_status lora_weight_amax(const qf_qlinear_desc* d, const qf::LoraOperand& L, const uint16_t* W,
                           int64_t ldw, float* scratch, const float** g, hipStream_t s) {
  *g = d->w_amax;
  if (d->wfmt != QF_FMT_NVFP4 || *g) return QF_OK;
  QF_TRY(dev(qf::launch_fill_f32(scratch, 1, 0.0f, s), "amax init"));
  QF_TRY(dev(qf::launch_lora_amax(L, W, d->N, d->K, ldw, 1, 0, scratch, s), "merged amax"));
  *g = scratch;
  return QF_OK;
}

// NVFP4 without a given amax needs the merged tensor's amax before any block scale.  Rather
// than merging twice (an amax pass, then the quantizer), the merged bf16 tensor m = bf16(W +
// scale B A) is written once to `tmp` [N, K] and the amax and the quantizer read it: the same m
// values through the same codec, so the output is bit-identical.  Transposed: out [K, N].
bool lora_merge_once(const qf_qlinear_desc* d) { return d->wfmt == QF_FMT_NVFP4 && !d->w_amax; }

qf_status lora_quant_via_merged(const qf_qlinear_desc* d, const qf::LoraOperand& L,
                                const uint16_t* W, int64_t ldw, uint16_t* tmp, float* scratch,
                                uint16_t* out, bool transposed, hipStream_t s) {
  const int64_t N = d->N, K = d->K;
  QF_TRY(dev(qf::launch_lora_quant(QF_FMT_NONE, L, W, N, K, ldw, 1, 0, nullptr, nullptr, nullptr,
                                   nullptr, nullptr, tmp, s),
             "merge"));
  QF_TRY(dev(qf::launch_amax(tmp, N, K, K, scratch, false, s), "amax of the merged weight"));
  if (transposed)
    QF_TRY(dev(qf::launch_quant_t(QF_FMT_NVFP4, tmp, N, K, K, 1, 0, scratch, out, N, 0, s),
               "quantize merged weight (transposed)"));
  else
    QF_TRY(dev(qf::launch_nvfp4(tmp, N, K, K, scratch, nullptr, nullptr, nullptr, out, s),
               "quantize merged weight"));
  return QF_OK;
}

}  // namespace

qf_status qf_lora_amax(const uint16_t* W, int64_t N, int64_t K, int64_t ldw, const qf_lora* lora,
                       float* amax, int accumulate, qf_stream_t stream) {
  const char* fn = "qf_lora_amax";
  QF_TRY(check_quant_input(fn, W, N, K, ldw, 8));
  QF_TRY(check_lora(fn, lora, N, K));
  if (!amax) return fail(QF_EINVAL, "%s: null amax", fn);
  if (accumulate != 0 && accumulate != 1) return fail(QF_EINVAL, "%s: accumulate must be 0/1", fn);
  hipStream_t s = S(stream);
  if (!accumulate) QF_TRY(dev(qf::launch_fill_f32(amax, 1, 0.0f, s), "amax init"));
  QF_TRY(dev(qf::launch_lora_amax(lora_op(lora), W, N, K, ldw, 1, 0, amax, s), "merged amax"));
  return ok();
}

qf_status qf_lora_fakequant(int fmt, const uint16_t* W, int64_t N, int64_t K, int64_t ldw,
                            const qf_lora* lora, float* amax, int amax_mode, float* s_out,
                            uint8_t* codes, uint8_t* scales, uint8_t* packed, uint16_t* xhat,
                            qf_stream_t stream) {
  const char* fn = "qf_lora_fakequant";
  if (!fmt_valid(fmt)) return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  QF_TRY(check_quant_input(fn, W, N, K, ldw, block_of(fmt)));
  QF_TRY(check_lora(fn, lora, N, K));
  const bool fp4 = fmt == QF_FMT_NVFP4 || fmt == QF_FMT_MXFP4;
  if ((codes || scales) && !fp4) return fail(QF_EINVAL, "%s: codes/scales are NVFP4/MXFP4 outputs", fn);
  if (packed && fmt != QF_FMT_Q4K) return fail(QF_EINVAL, "%s: packed is the Q4_K output", fn);
  QF_TRY(check_out("qf_lora_fakequant: codes", codes));
  QF_TRY(check_out("qf_lora_fakequant: scales", scales));
  QF_TRY(check_out("qf_lora_fakequant: packed", packed));
  QF_TRY(check_out("qf_lora_fakequant: xhat", xhat));
  hipStream_t s = S(stream);
  const qf::LoraOperand L = lora_op(lora);
  if (fmt == QF_FMT_NVFP4) {
    if (!amax) return fail(QF_EINVAL, "%s: NVFP4 needs amax", fn);
    if (amax_mode != QF_AMAX_COMPUTE && amax_mode != QF_AMAX_GIVEN)
      return fail(QF_EINVAL, "%s: bad amax_mode %d", fn, amax_mode);
    if (s_out && s_out == amax) return fail(QF_EINVAL, "%s: s_out aliases amax", fn);
    if (amax_mode == QF_AMAX_COMPUTE) {
      QF_TRY(dev(qf::launch_fill_f32(amax, 1, 0.0f, s), "amax init"));
      QF_TRY(dev(qf::launch_lora_amax(L, W, N, K, ldw, 1, 0, amax, s), "merged amax"));
    }
    if ((N == 0 || K == 0) && s_out) QF_TRY(dev(qf::launch_fill_f32(s_out, 1, 0.0f, s), "S"));
  } else if (s_out) {
    return fail(QF_EINVAL, "%s: s_out is an NVFP4 output", fn);
  }
  QF_TRY(dev(qf::launch_lora_quant(fmt, L, W, N, K, ldw, 1, 0, amax, s_out, codes, scales, packed,
                                   xhat, s),
             "merged quantize"));
  return ok();
}

qf_status qf_lora_fakequant_transposed(int fmt, const uint16_t* W, int64_t N, int64_t K,
                                       int64_t ldw, const qf_lora* lora, const float* amax,
                                       uint16_t* out, int64_t ldo, qf_stream_t stream) {
  const char* fn = "qf_lora_fakequant_transposed";
  if (!fmt_valid(fmt)) return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  QF_TRY(check_quant_input(fn, W, N, K, ldw, block_of(fmt)));
  QF_TRY(check_lora(fn, lora, N, K));
  if (N % 8) return fail(QF_ESHAPE, "%s: N=%lld is not a multiple of 8", fn, (long long)N);
  if (N == 0 || K == 0) return ok();
  if (fmt == QF_FMT_NVFP4 && !amax) return fail(QF_EINVAL, "%s: NVFP4 needs amax", fn);
  if (!out) return fail(QF_EINVAL, "%s: null output", fn);
  QF_TRY(check_mat("qf_lora_fakequant_transposed: out", out, K, N, ldo, true));
  QF_TRY(dev(qf::launch_lora_quant_t(fmt, lora_op(lora), W, N, K, ldw, 1, 0, amax, out, ldo, 0,
                                     S(stream)),
             "merged quantize (transposed)"));
  return ok();
}

qf_status qf_lora_workspace_size(const qf_qlinear_desc* d, const qf_lora* lora, size_t* bytes) {
  Dims dm;
  QF_TRY(check_desc("qf_lora_workspace_size", d, &dm));
  QF_TRY(check_lora("qf_lora_workspace_size", lora, 0, 0));
  if (!bytes) return fail(QF_EINVAL, "qf_lora_workspace_size: null output");
  *bytes = lora_ws_bytes(d, lora->r);
  return ok();
}

qf_status qf_qlinear_lora_fwd(const qf_qlinear_desc* d, const qf_lora* lora, const uint16_t* X,
                              const uint16_t* W, uint16_t* Y, void* ws, size_t ws_bytes,
                              qf_stream_t stream) {
  const char* fn = "qf_qlinear_lora_fwd";
  Dims dm;
  QF_TRY(check_desc(fn, d, &dm));
  QF_TRY(check_lora(fn, lora, d->N, d->K));
  QF_TRY(check_mat("qf_qlinear_lora_fwd: X", X, d->M, d->K, dm.ldx, true));
  QF_TRY(check_mat("qf_qlinear_lora_fwd: W", W, d->N, d->K, dm.ldw, true));
  QF_TRY(check_mat("qf_qlinear_lora_fwd: Y", Y, d->M, d->N, dm.ldy, true));
  QF_TRY(check_ws(fn, lora_ws_bytes(d, lora->r), ws, ws_bytes));
  hipStream_t s = S(stream);
  LoraWs w = lora_ws(d, lora->r, ws);
  const qf::LoraOperand L = lora_op(lora);
  if (lora_merge_once(d)) {           // W_hat^T's region is free in the forward
    QF_TRY(lora_quant_via_merged(d, L, W, dm.ldw, w.whatt, w.scal, w.what, false, s));
  } else {
    const float* g;
    QF_TRY(lora_weight_amax(d, L, W, dm.ldw, w.scal, &g, s));
    QF_TRY(dev(qf::launch_lora_quant(d->wfmt, L, W, d->N, d->K, dm.ldw, 1, 0, g, nullptr, nullptr,
                                     nullptr, nullptr, w.what, s),
               "merged quantize"));
  }
  const uint16_t* Aop = X;
  int64_t lda = dm.ldx;
  if (d->afmt != QF_FMT_NONE) {
    QF_TRY(fakequant_to(d->afmt, X, d->M, d->K, dm.ldx, d->a_amax, nullptr, w.ahat, s));
    Aop = w.ahat;
    lda = d->K;
  }
  QF_TRY(dev(qf::launch_gemm_nt(d->M, d->N, d->K, Aop, lda, 0, w.what, d->K, 0, Y, dm.ldy, 0,
                                nullptr, s),
             "forward gemm"));
  return ok();
}

qf_status qf_qlinear_lora_bwd_ste(const qf_qlinear_desc* d, const qf_lora* lora,
                                  const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                                  uint16_t* dX, float* dA, float* dB, void* ws, size_t ws_bytes,
                                  qf_stream_t stream) {
  const char* fn = "qf_qlinear_lora_bwd_ste";
  Dims dm;
  QF_TRY(check_desc(fn, d, &dm));
  QF_TRY(check_lora(fn, lora, d->N, d->K));
  const bool grads = dA || dB;
  QF_TRY(check_mat("qf_qlinear_lora_bwd_ste: dY", dY, d->M, d->N, dm.ldy, true));
  QF_TRY(check_mat("qf_qlinear_lora_bwd_ste: X", X, d->M, d->K, dm.ldx, grads));
  QF_TRY(check_mat("qf_qlinear_lora_bwd_ste: W", W, d->N, d->K, dm.ldw, dX != nullptr));
  QF_TRY(check_mat("qf_qlinear_lora_bwd_ste: dX", dX, d->M, d->K, dm.ldx, false));
  QF_TRY(check_out("qf_qlinear_lora_bwd_ste: dA", dA));
  QF_TRY(check_out("qf_qlinear_lora_bwd_ste: dB", dB));
  QF_TRY(check_ws(fn, lora_ws_bytes(d, lora->r), ws, ws_bytes));
  hipStream_t s = S(stream);
  LoraWs w = lora_ws(d, lora->r, ws);
  const qf::LoraOperand L = lora_op(lora);
  const bool reuse = (d->flags & QF_FLAG_REUSE_WS) != 0;
  const int64_t M = d->M, N = d->N, K = d->K, r = lora->r, rp = (r + 15) / 16 * 16;
  if (dX && M > 0 && K > 0) {  // dX[M, K] = dY[M, N] (W_hat^T)[K, N]^T
    if (reuse) {
      QF_TRY(dev(qf::launch_transpose_bf16(w.what, N, K, K, w.whatt, N, 1, 0, 0, s),
                 "transpose W_hat"));
    } else if (lora_merge_once(d)) {    // W_hat's region is free without a saved forward
      QF_TRY(lora_quant_via_merged(d, L, W, dm.ldw, w.what, w.scal, w.whatt, true, s));
    } else {
      const float* g;
      QF_TRY(lora_weight_amax(d, L, W, dm.ldw, w.scal, &g, s));
      QF_TRY(dev(qf::launch_lora_quant_t(d->wfmt, L, W, N, K, dm.ldw, 1, 0, g, w.whatt, N, 0, s),
                 "merged quantize (transposed)"));
    }
    QF_TRY(dev(qf::launch_gemm_nt(M, K, N, dY, dm.ldy, 0, w.whatt, N, 0, dX, dm.ldx, 0, nullptr,
                                  s),
               "dX gemm"));
  }
  if (!grads) return ok();
  const uint16_t* Aop = X;
  int64_t lda = dm.ldx;
  if (d->afmt != QF_FMT_NONE) {
    if (!reuse && M > 0)
      QF_TRY(fakequant_to(d->afmt, X, M, K, dm.ldx, d->a_amax, nullptr, w.ahat, s));
    Aop = w.ahat;
    lda = K;
  }
  if (dB) {  // dB = scale dY^T (A_hat A^T)
    QF_TRY(dev(qf::launch_lora_rowdot(Aop, M, K, lda, L.A, K, r, w.u, rp, nullptr, nullptr, 0, 0, s), "A_hat A^T"));
    QF_TRY(dev(qf::launch_lora_colsum(dY, M, N, dm.ldy, w.u, rp, r, L.scale, w.part, 0, dB, nullptr,
                                          nullptr, 0, 0, s),
               "dB"));
  }
  if (dA) {  // dA = scale (dY B)^T A_hat
    QF_TRY(dev(qf::launch_transpose_f32(L.B, N, r, 1, w.bt, s), "B^T"));
    QF_TRY(dev(qf::launch_lora_rowdot(dY, M, N, dm.ldy, w.bt, N, r, w.v, rp, nullptr, nullptr, 0, 0, s), "dY B"));
    QF_TRY(dev(qf::launch_lora_colsum(Aop, M, K, lda, w.v, rp, r, L.scale, w.part, 1, dA, nullptr,
                                          nullptr, 0, 0, s),
               "dA"));
  }
  return ok();
}

// -------------------------------------------------------------------- grouped LoRA-QAD (MoE)
namespace {

// Workspace of the grouped LoRA layer (256-byte aligned regions):
//   tile_start, order  [E+1], [E]   grouped NT row tiles (launch_grouped_prep)
//   pre16, prech       [E+1] x 2    row-dot / column-sum chunk prefixes
//   wamax              [E]          per-expert merged amax (NVFP4)
//   what               [E, N, K]    per-expert W_hat of the merged weights
//   ahat               [T, K]       A_hat (afmt MXFP4)
//   whatt              [E, K, N]    per-expert W_hat^T (dX operand in NT form)
//   bt                 [Eb, r, N]   B^T per expert (Eb = 1 when B is shared)
//   u, v               [T, rp]      A_hat A_e^T and dY B_e (FP32)
//   part                            column-sum chunk partials
struct GroupedLoraWs {
  int* tile_start;
  int* order;
  int* pre16;
  int* prech;
  float* wamax;
  uint16_t* what;
  uint16_t* ahat;
  uint16_t* whatt;
  float* bt;
  float* u;
  float* v;
  float* part;
};

size_t glora_ws_bytes(const qf_grouped_desc* d, int64_t r, int b_shared) {
  const size_t E = d->E, T = d->T, N = d->N, K = d->K, R = r, RP = (R + 15) / 16 * 16;
  const size_t Eb = b_shared ? 1 : E;
  size_t b = up((E + 1) * 4) + up(E * 4) + 2 * up((E + 1) * 4) + up(E * 4);
  b += up(E * N * K * 2);
  if (d->afmt != QF_FMT_NONE) b += up(T * K * 2);
  b += up(E * K * N * 2) + up(Eb * R * N * 4) + 2 * up(T * RP * 4);
  const size_t p1 = qf::lora_colsum_grouped_part_bytes(d->T, d->E, d->N, r);
  const size_t p2 = qf::lora_colsum_grouped_part_bytes(d->T, d->E, d->K, r);
  return b + up(p1 > p2 ? p1 : p2);
}

GroupedLoraWs glora_ws(const qf_grouped_desc* d, int64_t r, int b_shared, void* ws) {
  const size_t E = d->E, T = d->T, N = d->N, K = d->K, R = r, RP = (R + 15) / 16 * 16;
  const size_t Eb = b_shared ? 1 : E;
  char* p = static_cast<char*>(ws);
  GroupedLoraWs g{};
  g.tile_start = reinterpret_cast<int*>(p); p += up((E + 1) * 4);
  g.order = reinterpret_cast<int*>(p); p += up(E * 4);
  g.pre16 = reinterpret_cast<int*>(p); p += up((E + 1) * 4);
  g.prech = reinterpret_cast<int*>(p); p += up((E + 1) * 4);
  g.wamax = reinterpret_cast<float*>(p); p += up(E * 4);
  g.what = reinterpret_cast<uint16_t*>(p); p += up(E * N * K * 2);
  if (d->afmt != QF_FMT_NONE) { g.ahat = reinterpret_cast<uint16_t*>(p); p += up(T * K * 2); }
  g.whatt = reinterpret_cast<uint16_t*>(p); p += up(E * K * N * 2);
  g.bt = reinterpret_cast<float*>(p); p += up(Eb * R * N * 4);
  g.u = reinterpret_cast<float*>(p); p += up(T * RP * 4);
  g.v = reinterpret_cast<float*>(p); p += up(T * RP * 4);
  g.part = reinterpret_cast<float*>(p);
  return g;
}

qf_status check_glora(const char* fn, const qf_grouped_desc* d, const int64_t* off,
                      const qf_lora* L) {
  QF_TRY(check_grouped(fn, d, off));
  QF_TRY(check_lora(fn, L, d->N, d->K));
  if ((L->a_shared & ~1) || (L->b_shared & ~1))
    return fail(QF_EINVAL, "%s: a_shared / b_shared must be 0 or 1", fn);
  return QF_OK;
}

qf::LoraOperand glora_op(const qf_grouped_desc* d, const qf_lora* L) {
  return qf::LoraOperand{L->A, L->a_shared ? 0 : L->r * d->K, L->B,
                         L->b_shared ? 0 : d->N * L->r, L->r, L->scale};
}

// Per-expert NVFP4 amax of the merged weights (or the caller's tied values).
qf_status glora_amax(const qf_grouped_desc* d, const qf::LoraOperand& L, const uint16_t* W,
                     float* scratch, const float** g, hipStream_t s) {
  *g = d->w_amax;
  if (d->wfmt != QF_FMT_NVFP4 || *g) return QF_OK;
  QF_TRY(dev(qf::launch_fill_f32(scratch, d->E, 0.0f, s), "amax init"));
  QF_TRY(dev(qf::launch_lora_amax(L, W, d->N, d->K, d->K, d->E, d->N * d->K, scratch, s),
             "merged amax"));
  *g = scratch;
  return QF_OK;
}

// As lora_quant_via_merged, per expert: the merged experts go to `tmp` [E, N, K] once, then the
// per-expert amax and NVFP4 quantizer (row-major into out [E, N, K], or transposed into
// out [E, K, N]) read them.
bool glora_merge_once(const qf_grouped_desc* d) { return d->wfmt == QF_FMT_NVFP4 && !d->w_amax; }

qf_status glora_quant_via_merged(const qf_grouped_desc* d, const qf::LoraOperand& L,
                                 const uint16_t* W, uint16_t* tmp, float* scratch, uint16_t* out,
                                 bool transposed, hipStream_t s) {
  const int64_t E = d->E, N = d->N, K = d->K;
  QF_TRY(dev(qf::launch_lora_quant(QF_FMT_NONE, L, W, N, K, K, E, N * K, nullptr, nullptr,
                                   nullptr, nullptr, nullptr, tmp, s),
             "merge (experts)"));
  QF_TRY(dev(qf::launch_amax_batched(tmp, E, N, K, scratch, false, s), "amax of the merged experts"));
  if (transposed)
    QF_TRY(dev(qf::launch_quant_t(QF_FMT_NVFP4, tmp, N, K, K, E, N * K, scratch, out, N, N * K, s),
               "quantize merged experts (transposed)"));
  else
    QF_TRY(dev(qf::launch_nvfp4_batched(tmp, E, N, K, scratch, nullptr, nullptr, nullptr, out, s),
               "quantize merged experts"));
  return QF_OK;
}

}  // namespace

qf_status qf_grouped_lora_workspace_size(const qf_grouped_desc* d, const qf_lora* lora,
                                         size_t* bytes) {
  QF_TRY(check_glora("qf_grouped_lora_workspace_size", d, (const int64_t*)1, lora));
  if (!bytes) return fail(QF_EINVAL, "qf_grouped_lora_workspace_size: null output");
  *bytes = glora_ws_bytes(d, lora->r, lora->b_shared);
  return ok();
}

qf_status qf_qlinear_grouped_lora_fwd(const qf_grouped_desc* d, const qf_lora* lora,
                                      const int64_t* group_offsets, const uint16_t* X,
                                      const uint16_t* W, uint16_t* Y, void* ws, size_t ws_bytes,
                                      qf_stream_t stream) {
  const char* fn = "qf_qlinear_grouped_lora_fwd";
  QF_TRY(check_glora(fn, d, group_offsets, lora));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_fwd: X", X, d->T, d->K, d->K, true));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_fwd: W", W, d->E * d->N, d->K, d->K, true));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_fwd: Y", Y, d->T, d->N, d->N, true));
  QF_TRY(check_ws(fn, glora_ws_bytes(d, lora->r, lora->b_shared), ws, ws_bytes));
  if (d->E == 0) return ok();
  hipStream_t s = S(stream);
  GroupedLoraWs g = glora_ws(d, lora->r, lora->b_shared, ws);
  const qf::LoraOperand L = glora_op(d, lora);
  if (glora_merge_once(d)) {          // the experts' W_hat^T region is free in the forward
    QF_TRY(glora_quant_via_merged(d, L, W, g.whatt, g.wamax, g.what, false, s));
  } else {
    const float* gp;
    QF_TRY(glora_amax(d, L, W, g.wamax, &gp, s));
    QF_TRY(dev(qf::launch_lora_quant(d->wfmt, L, W, d->N, d->K, d->K, d->E, d->N * d->K, gp,
                                     nullptr, nullptr, nullptr, nullptr, g.what, s),
               "merged quantize (experts)"));
  }
  const uint16_t* Aop = X;
  if (d->afmt == QF_FMT_MXFP4) {
    QF_TRY(dev(qf::launch_mxfp4(X, d->T, d->K, d->K, nullptr, nullptr, g.ahat, s), "mxfp4"));
    Aop = g.ahat;
  }
  QF_TRY(dev(qf::launch_grouped_prep(group_offsets, d->E, g.tile_start, g.order, nullptr, s),
             "prep"));
  QF_TRY(dev(qf::launch_grouped_nt_rows(d->E, d->T, d->N, d->K, group_offsets, g.tile_start, Aop,
                                        d->K, g.what, d->K, 0, d->N * d->K, Y, d->N, s),
             "grouped forward"));
  return ok();
}

qf_status qf_qlinear_grouped_lora_bwd_ste(const qf_grouped_desc* d, const qf_lora* lora,
                                          const int64_t* group_offsets, const uint16_t* dY,
                                          const uint16_t* X, const uint16_t* W, uint16_t* dX,
                                          float* dA, float* dB, void* ws, size_t ws_bytes,
                                          qf_stream_t stream) {
  const char* fn = "qf_qlinear_grouped_lora_bwd_ste";
  QF_TRY(check_glora(fn, d, group_offsets, lora));
  const bool grads = dA || dB;
  QF_TRY(check_mat("qf_qlinear_grouped_lora_bwd_ste: dY", dY, d->T, d->N, d->N, true));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_bwd_ste: X", X, d->T, d->K, d->K, grads));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_bwd_ste: W", W, d->E * d->N, d->K, d->K, dX != nullptr));
  QF_TRY(check_mat("qf_qlinear_grouped_lora_bwd_ste: dX", dX, d->T, d->K, d->K, false));
  QF_TRY(check_out("qf_qlinear_grouped_lora_bwd_ste: dA", dA));
  QF_TRY(check_out("qf_qlinear_grouped_lora_bwd_ste: dB", dB));
  QF_TRY(check_ws(fn, glora_ws_bytes(d, lora->r, lora->b_shared), ws, ws_bytes));
  if (d->E == 0) return ok();
  hipStream_t s = S(stream);
  GroupedLoraWs g = glora_ws(d, lora->r, lora->b_shared, ws);
  const qf::LoraOperand L = glora_op(d, lora);
  const bool reuse = (d->flags & QF_FLAG_REUSE_WS) != 0;
  const int64_t E = d->E, T = d->T, N = d->N, K = d->K, r = lora->r, rp = (r + 15) / 16 * 16;
  if (dX) {
    QF_TRY(dev(qf::launch_grouped_prep(group_offsets, E, g.tile_start, g.order, nullptr, s),
               "prep"));
    if (reuse) {
      QF_TRY(dev(qf::launch_transpose_bf16(g.what, N, K, K, g.whatt, N, E, N * K, N * K, s),
                 "transpose expert W_hat"));
    } else if (glora_merge_once(d)) {   // W_hat's region is free without a saved forward
      QF_TRY(glora_quant_via_merged(d, L, W, g.what, g.wamax, g.whatt, true, s));
    } else {
      const float* gp;
      QF_TRY(glora_amax(d, L, W, g.wamax, &gp, s));
      QF_TRY(dev(qf::launch_lora_quant_t(d->wfmt, L, W, N, K, K, E, N * K, gp, g.whatt, N, N * K,
                                         s),
                 "merged quantize (experts, transposed)"));
    }
    QF_TRY(dev(qf::launch_grouped_nt_rows(E, T, K, N, group_offsets, g.tile_start, dY, N, g.whatt,
                                          N, 0, N * K, dX, K, s),
               "grouped dX"));
  }
  if (!grads) return ok();
  const uint16_t* Aop = X;
  if (d->afmt == QF_FMT_MXFP4) {
    if (!reuse && T > 0)
      QF_TRY(dev(qf::launch_mxfp4(X, T, K, K, nullptr, nullptr, g.ahat, s), "mxfp4"));
    Aop = g.ahat;
  }
  QF_TRY(dev(qf::launch_group_prefix(group_offsets, E, 16, g.pre16, s), "row prefix"));
  QF_TRY(dev(qf::launch_group_prefix(group_offsets, E, 1024, g.prech, s), "chunk prefix"));
  if (dB) {  // dB_e = scale dY_e^T (A_hat_e A_e^T); shared B: summed over experts
    QF_TRY(dev(qf::launch_lora_rowdot(Aop, T, K, K, L.A, K, r, g.u, rp, group_offsets, g.pre16, E,
                                      L.a_stride, s),
               "A_hat A_e^T"));
    QF_TRY(dev(qf::launch_lora_colsum(dY, T, N, N, g.u, rp, r, L.scale, g.part, 0, dB,
                                      group_offsets, g.prech, E, !lora->b_shared, s),
               "dB"));
  }
  if (dA) {  // dA_e = scale (dY_e B_e)^T A_hat_e; shared A: summed over experts
    QF_TRY(dev(qf::launch_transpose_f32(L.B, N, r, lora->b_shared ? 1 : E, g.bt, s), "B^T"));
    QF_TRY(dev(qf::launch_lora_rowdot(dY, T, N, N, g.bt, N, r, g.v, rp, group_offsets, g.pre16, E,
                                      lora->b_shared ? 0 : r * N, s),
               "dY B_e"));
    QF_TRY(dev(qf::launch_lora_colsum(Aop, T, K, K, g.v, rp, r, L.scale, g.part, 1, dA,
                                      group_offsets, g.prech, E, !lora->a_shared, s),
               "dA"));
  }
  return ok();
}

// ------------------------------------------------------------------ QAD distillation loss
qf_status qf_qad_kl(const uint16_t* zt, int64_t ldt, const uint16_t* zs, int64_t lds, int64_t L,
                    int64_t V, float grad_scale, float* row_kl, float* loss, uint16_t* grad,
                    int64_t ldg, int32_t* agree, qf_stream_t stream) {
  const char* fn = "qf_qad_kl";
  if (L < 0 || V < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (V % 8) return fail(QF_ESHAPE, "%s: V=%lld is not a multiple of 8", fn, (long long)V);
  if (L > 0 && V == 0) return fail(QF_ESHAPE, "%s: empty vocabulary", fn);
  QF_TRY(check_mat("qf_qad_kl: zt", zt, L, V, ldt, true));
  QF_TRY(check_mat("qf_qad_kl: zs", zs, L, V, lds, true));
  QF_TRY(check_mat("qf_qad_kl: grad", grad, L, V, ldg, false));
  if (L > 0 && !row_kl) return fail(QF_EINVAL, "%s: null row_kl", fn);
  QF_TRY(check_out("qf_qad_kl: agree", agree));
  QF_TRY(dev(qf::launch_qad_kl(zt, ldt, zs, lds, L, V, grad_scale, row_kl, loss, grad, ldg, agree,
                               S(stream)),
             "qad kl"));
  return ok();
}

// --------------------------------------------------------------- engine-native export / sync
namespace {

constexpr uint32_t kPayloadMagic = 0x31504651u;   // "QFP1"

qf_status payload_layout(int fmt, int64_t N, int64_t K, qf_payload_layout* L) {
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4)
    return fail(QF_EINVAL, "payload: format must be NVFP4 or MXFP4");
  if (N < 0 || K < 0) return fail(QF_ESHAPE, "payload: negative shape");
  const int64_t blk = block_of(fmt);
  if (K % blk) return fail(QF_ESHAPE, "payload: K=%lld is not a multiple of %lld", (long long)K,
                           (long long)blk);
  L->codes = 256;
  L->scales = L->codes + up((size_t)N * K / 2);
  L->scalars = L->scales + up((size_t)N * K / blk);
  L->total = L->scalars + 256;
  return QF_OK;
}

}  // namespace

qf_status qf_payload_layout_of(int fmt, int64_t N, int64_t K, qf_payload_layout* out) {
  if (!out) return fail(QF_EINVAL, "qf_payload_layout_of: null output");
  QF_TRY(payload_layout(fmt, N, K, out));
  return ok();
}

qf_status qf_payload_write_header(int fmt, int64_t N, int64_t K, void* payload,
                                  qf_stream_t stream) {
  qf_payload_layout L;
  QF_TRY(payload_layout(fmt, N, K, &L));
  if (!payload) return fail(QF_EINVAL, "qf_payload_write_header: null payload");
  if ((uintptr_t)payload % kAlign)
    return fail(QF_EALIGN, "qf_payload_write_header: payload not 256-byte aligned");
  const uint64_t q[7] = {(uint64_t)N, (uint64_t)K, L.codes, L.scales, L.scalars, L.total, 0};
  uint32_t w[16];
  w[0] = kPayloadMagic;
  w[1] = (uint32_t)fmt;
  for (int i = 0; i < 7; ++i) {
    w[2 + 2 * i] = (uint32_t)(q[i] & 0xFFFFFFFFu);
    w[3 + 2 * i] = (uint32_t)(q[i] >> 32);
  }
  QF_TRY(dev(qf::launch_payload_header(payload, w, S(stream)), "payload header"));
  return ok();
}

qf_status qf_export_fused(int fmt, const qf_member* members, int n, int64_t K, uint8_t* codes,
                          uint8_t* scales, float* w_amax, float* weight_scale_2,
                          const float* a_amax, float* input_scale, qf_stream_t stream) {
  const char* fn = "qf_export_fused";
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4)
    return fail(QF_EINVAL, "%s: format must be NVFP4 or MXFP4", fn);
  if (!members || n < 1 || n > 8) return fail(QF_EINVAL, "%s: 1 to 8 members", fn);
  const int64_t blk = block_of(fmt);
  int64_t N = 0;
  for (int i = 0; i < n; ++i) {
    QF_TRY(check_quant_input(fn, members[i].W, members[i].rows, K, members[i].ldw, blk));
    N += members[i].rows;
  }
  if (!codes || !scales) return fail(QF_EINVAL, "%s: codes and scales are required", fn);
  QF_TRY(check_out("qf_export_fused: codes", codes));
  hipStream_t s = S(stream);
  if (fmt == QF_FMT_NVFP4) {
    if (!w_amax) return fail(QF_EINVAL, "%s: NVFP4 needs w_amax", fn);
    if (input_scale && !a_amax) return fail(QF_EINVAL, "%s: input_scale needs a_amax", fn);
    for (int i = 0; i < n; ++i)       // the first member sets g, the others fold into it
      QF_TRY(dev(qf::launch_amax(members[i].W, members[i].rows, K, members[i].ldw, w_amax,
                                 i > 0, s),
                 "tied amax"));
    int64_t r0 = 0;
    for (int i = 0; i < n; ++i) {
      QF_TRY(dev(qf::launch_nvfp4(members[i].W, members[i].rows, K, members[i].ldw, w_amax,
                                  nullptr, codes + r0 * (K / 2), scales + r0 * (K / 16), nullptr,
                                  s),
                 "nvfp4 member"));
      r0 += members[i].rows;
    }
    if (weight_scale_2 || input_scale)
      QF_TRY(dev(qf::launch_export_scalars(w_amax, a_amax, weight_scale_2, input_scale, s),
                 "export scalars"));
  } else {
    if (w_amax || weight_scale_2 || input_scale)
      return fail(QF_EINVAL, "%s: MXFP4 has no tensor-level scales", fn);
    int64_t r0 = 0;
    for (int i = 0; i < n; ++i) {
      QF_TRY(dev(qf::launch_mxfp4(members[i].W, members[i].rows, K, members[i].ldw,
                                  codes + r0 * (K / 2), scales + r0 * (K / 32), nullptr, s),
                 "mxfp4 member"));
      r0 += members[i].rows;
    }
  }
  (void)N;
  return ok();
}

// ------------------------------------------------------------- fragment-major B operands
qf_status qf_fragment_bytes(int64_t N, int64_t K, size_t* bytes) {
  if (N < 0 || K < 0) return fail(QF_ESHAPE, "qf_fragment_bytes: negative shape");
  if (K % 16) return fail(QF_ESHAPE, "qf_fragment_bytes: K=%lld is not a multiple of 16", (long long)K);
  if (!bytes) return fail(QF_EINVAL, "qf_fragment_bytes: null output");
  *bytes = qf::gemm_frag_bytes(N, K);
  return ok();
}

qf_status qf_pack_fragments(const uint16_t* B, int64_t N, int64_t K, int64_t ldb, uint16_t* out,
                            qf_stream_t stream) {
  const char* fn = "qf_pack_fragments";
  if (N < 0 || K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (K % 16) return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of 16", fn, (long long)K);
  QF_TRY(check_mat("qf_pack_fragments: B", B, N, K, ldb, true));
  if (N == 0 || K == 0) return ok();
  if (!out) return fail(QF_EINVAL, "%s: null output", fn);
  QF_TRY(check_out("qf_pack_fragments: out", out));
  QF_TRY(dev(qf::launch_frag_pack(B, N, K, ldb, out, S(stream)), fn));
  return ok();
}

qf_status qf_gemm_bf16_fragb(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                             const uint16_t* Bf, void* C, int64_t ldc, int c_f32, void* ws,
                             size_t ws_bytes, qf_stream_t stream) {
  const char* fn = "qf_gemm_bf16_fragb";
  if (M < 0 || N < 0 || K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (K % 64) return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of 64", fn, (long long)K);
  if (c_f32 != 0 && c_f32 != 1) return fail(QF_EINVAL, "%s: c_f32 must be 0/1", fn);
  QF_TRY(check_mat("qf_gemm_bf16_fragb: A", A, M, K, lda, true));
  if (!C && M > 0 && N > 0) return fail(QF_EINVAL, "%s: null C", fn);
  if (ldc < N) return fail(QF_ESHAPE, "%s: ldc < N", fn);
  if (M == 0 || N == 0) return ok();
  if (!Bf) return fail(QF_EINVAL, "%s: null B", fn);
  QF_TRY(check_out("qf_gemm_bf16_fragb: B", Bf));
  float* part = nullptr;
  if (c_f32 && ws) {
    if ((uintptr_t)ws % kAlign) return fail(QF_EALIGN, "%s: workspace not 256-byte aligned", fn);
    if (ws_bytes >= qf::gemm_nt_split_bytes(M, N)) part = static_cast<float*>(ws);
  }
  QF_TRY(dev(qf::launch_gemm_nt_bf(M, N, K, A, lda, Bf, C, ldc, c_f32, part, S(stream)), fn));
  return ok();
}

// ---------------------------------------------------------- packed-operand building blocks
qf_status qf_gemm_packed_b(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                           int fmt, const uint8_t* codes, const uint8_t* scales, const float* Sp,
                           uint16_t* C, int64_t ldc, qf_stream_t stream) {
  const char* fn = "qf_gemm_packed_b";
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4 && fmt != QF_FMT_Q4K)
    return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  if (M < 0 || N < 0 || K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (K % (fmt == QF_FMT_Q4K ? 256 : 64))
    return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of %d", fn, (long long)K,
                fmt == QF_FMT_Q4K ? 256 : 64);
  QF_TRY(check_mat("qf_gemm_packed_b: A", A, M, K, lda, true));
  QF_TRY(check_mat("qf_gemm_packed_b: C", C, M, N, ldc, true));
  if (M == 0 || N == 0) return ok();
  if (!codes || (fmt != QF_FMT_Q4K && !scales) || (fmt == QF_FMT_NVFP4 && !Sp))
    return fail(QF_EINVAL, "%s: null packed operand", fn);
  QF_TRY(check_out("qf_gemm_packed_b: codes", codes));
  QF_TRY(check_out("qf_gemm_packed_b: scales", scales));
  QF_TRY(dev(qf::launch_gemm_nt_packed_b(M, N, K, A, lda, fmt, codes, scales, Sp, C, ldc,
                                         S(stream)), fn));
  return ok();
}

qf_status qf_dequantize_transposed(int fmt, const uint8_t* codes, const uint8_t* scales,
                                   const float* Sp, int64_t R, int64_t K, uint16_t* out,
                                   int64_t ldo, qf_stream_t stream) {
  const char* fn = "qf_dequantize_transposed";
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4 && fmt != QF_FMT_Q4K)
    return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  if (R < 0 || K < 0) return fail(QF_ESHAPE, "%s: negative shape", fn);
  if (K % block_of(fmt)) return fail(QF_ESHAPE, "%s: K=%lld is not a multiple of %lld", fn,
                                     (long long)K, (long long)block_of(fmt));
  if (R % 8) return fail(QF_ESHAPE, "%s: R=%lld is not a multiple of 8", fn, (long long)R);
  if (R == 0 || K == 0) return ok();
  if (!codes || (fmt != QF_FMT_Q4K && !scales) || (fmt == QF_FMT_NVFP4 && !Sp))
    return fail(QF_EINVAL, "%s: null packed operand", fn);
  QF_TRY(check_out("qf_dequantize_transposed: codes", codes));
  QF_TRY(check_mat("qf_dequantize_transposed: out", out, K, R, ldo, true));
  QF_TRY(dev(qf::launch_dequant_t(fmt, codes, scales, Sp, R, K, out, ldo, S(stream)), fn));
  return ok();
}

// ------------------------------------------------------------------- host-only validation
qf_status qf_validate_fakequant(int fmt, const void* x, int64_t R, int64_t K, int64_t ldx) {
  const char* fn = "qf_validate_fakequant";
  if (fmt != QF_FMT_NVFP4 && fmt != QF_FMT_MXFP4 && fmt != QF_FMT_Q4K)
    return fail(QF_EINVAL, "%s: bad format %d", fn, fmt);
  QF_TRY(check_quant_input(fn, static_cast<const uint16_t*>(x), R, K, ldx, block_of(fmt)));
  return ok();
}

qf_status qf_validate_qlinear(const qf_qlinear_desc* d, const void* X, const void* W,
                              const void* Y, const void* saved, const void* ws, size_t ws_bytes) {
  const char* fn = "qf_validate_qlinear";
  Dims dm;
  QF_TRY(check_desc(fn, d, &dm));
  QF_TRY(check_mat("qf_validate_qlinear: X", X, d->M, d->K, dm.ldx, true));
  QF_TRY(check_mat("qf_validate_qlinear: W", W, d->N, d->K, dm.ldw, true));
  QF_TRY(check_mat("qf_validate_qlinear: Y", Y, d->M, d->N, dm.ldy, true));
  QF_TRY(check_saved(fn, saved));
  QF_TRY(check_ws(fn, linear_ws_bytes(d), const_cast<void*>(ws), ws_bytes));
  return ok();
}

qf_status qf_validate_grouped(const qf_grouped_desc* d, const void* X, const void* W,
                              const void* Y, const void* saved, const void* ws,
                              size_t ws_bytes) {
  const char* fn = "qf_validate_grouped";
  // (the device offsets are the call's own argument; only their presence is checked there)
  static const int64_t kOffsetsPresent = 0;
  QF_TRY(check_grouped(fn, d, &kOffsetsPresent));
  QF_TRY(check_mat("qf_validate_grouped: X", X, d->T, d->K, d->K, true));
  QF_TRY(check_mat("qf_validate_grouped: W", W, d->E * d->N, d->K, d->K, true));
  QF_TRY(check_mat("qf_validate_grouped: Y", Y, d->T, d->N, d->N, true));
  QF_TRY(check_saved(fn, saved));
  QF_TRY(check_ws(fn, grouped_ws_bytes(d), const_cast<void*>(ws), ws_bytes));
  return ok();
}

}  // extern "C"

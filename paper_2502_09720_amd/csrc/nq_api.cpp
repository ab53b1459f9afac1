// C ABI of libnestquant.so: argument checking and dispatch to the kernels.
// The declarations and their contracts are in include/nestquant.h.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>

#include "nestquant.h"
#include "nq_kernels.hpp"

namespace {

thread_local char g_last_error[512] = "";

nq_status fail(nq_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

nq_status ok() {
  g_last_error[0] = '\0';
  return NQ_OK;
}

// Kernel attributes (the dynamic LDS limit) belong to each device: set them once on every
// device that a call's stream runs on, before its first launch there.
class PerDevice {
 public:
  explicit PerDevice(hipError_t (*fn)()) : fn_(fn) {}
  hipError_t ensure(hipStream_t st) {
    hipDevice_t dev = 0;
    hipError_t e = hipStreamGetDevice(st, &dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kDevices) return hipErrorInvalidDevice;
    if (done_[dev].load(std::memory_order_acquire)) return hipSuccess;
    std::lock_guard<std::mutex> g(mu_);
    if (done_[dev].load(std::memory_order_relaxed)) return hipSuccess;
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    const hipError_t r = fn_();
    if (cur != dev && (e = hipSetDevice(cur)) != hipSuccess) return e;
    if (r == hipSuccess) done_[dev].store(true, std::memory_order_release);
    return r;
  }

 private:
  static constexpr int kDevices = 64;
  hipError_t (*fn_)();
  std::mutex mu_;
  std::atomic<bool> done_[kDevices] = {};
};

constexpr int64_t kMaxCols = 65536;
constexpr int64_t kMaxRows = (int64_t)1 << 31;

nq_status check_params(const nq_params* p, int64_t cols, const char* who) {
  if (!p) return fail(NQ_ERR_INVALID_ARG, "%s: params is NULL", who);
  if (p->q < 2 || p->q > 16) return fail(NQ_ERR_INVALID_ARG, "%s: q=%d outside [2,16]", who, p->q);
  if (p->k < 1 || p->k > 4) return fail(NQ_ERR_INVALID_ARG, "%s: k=%d outside [1,4]", who, p->k);
  if (!std::isfinite(p->base) || !(p->base > 0.0))
    return fail(NQ_ERR_INVALID_ARG, "%s: base must be finite and > 0", who);
  if (p->decoder != NQ_DECODER_FULL && p->decoder != NQ_DECODER_M)
    return fail(NQ_ERR_INVALID_ARG, "%s: decoder=%d is not an nq_decoder", who, p->decoder);
  if (p->strategy != NQ_FIRST_BETA && p->strategy != NQ_OPT_BETA)
    return fail(NQ_ERR_INVALID_ARG, "%s: strategy=%d is not an nq_strategy", who, p->strategy);
  if (p->mult[0] != 0) {
    for (int t = 0; t < 4; ++t) {
      const int m = p->mult[t];
      if (t < p->k ? (m < 1 || m > 64 || (t > 0 && m <= p->mult[t - 1])) : m != 0)
        return fail(NQ_ERR_INVALID_ARG,
                    "%s: mult must be all zero, or k increasing integers in [1, 64] followed by "
                    "zeros", who);
    }
  } else if (p->mult[1] != 0 || p->mult[2] != 0 || p->mult[3] != 0) {
    return fail(NQ_ERR_INVALID_ARG, "%s: mult[0] = 0 needs the whole table zero", who);
  }
  if (std::sqrt((double)cols) / p->base >= 2097152.0)
    return fail(NQ_ERR_INVALID_ARG, "%s: base too small for cols=%lld (sqrt(cols)/base >= 2^21)",
                who, (long long)cols);
  return NQ_OK;
}

nq_status check_cols(int64_t cols, const char* who) {
  if (cols < 8 || cols % 8 != 0 || cols > kMaxCols)
    return fail(NQ_ERR_INVALID_ARG, "%s: cols=%lld must be a multiple of 8 in [8, %lld]", who,
                (long long)cols, (long long)kMaxCols);
  return NQ_OK;
}

size_t dtype_size(nq_dtype d) { return d == NQ_F32 ? 4 : 2; }

// The multiple of base for beta index i (0..3): the table, the uniform grid i + 1 when it
// is zero, and the largest beta for indices past k (never written by the encoder).
int beta_mult(const nq_params* p, int i) {
  if (p->mult[0] == 0) return i + 1;
  return p->mult[i < p->k ? i : p->k - 1];
}
uint32_t mult_table(const nq_params* p) {
  uint32_t t = 0;
  for (int i = 0; i < 4; ++i) t |= (uint32_t)beta_mult(p, i) << (8 * i);
  return t;
}
// Largest |m X2| of the operand's tiles: 2q times its largest multiple.
int tile_bound(const nq_params* p) { return 2 * p->q * beta_mult(p, p->k - 1); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

nq_status hip_status(hipError_t e, const char* who) {
  if (e != hipSuccess) return fail(NQ_ERR_HIP, "%s: %s", who, hipGetErrorString(e));
  return ok();
}

}  // namespace

namespace nq {
nq_status set_error(nq_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}
}  // namespace nq

extern "C" {

int64_t nq_codes_words(int64_t rows, int64_t cols) {
  if (rows < 0 || cols < 8 || cols % 8) return -1;
  return rows * (cols / 8);
}

int64_t nq_beta_words(int64_t rows, int64_t cols) {
  if (rows < 0 || cols < 8 || cols % 8) return -1;
  return rows * ((cols / 8 + 15) / 16);
}

const char* nq_status_string(nq_status s) {
  switch (s) {
    case NQ_OK: return "NQ_OK";
    case NQ_ERR_INVALID_ARG: return "NQ_ERR_INVALID_ARG: invalid argument";
    case NQ_ERR_UNSUPPORTED: return "NQ_ERR_UNSUPPORTED: unsupported configuration";
    case NQ_ERR_HIP: return "NQ_ERR_HIP: HIP runtime error";
    default: break;
  }
  return "unknown nq_status";
}

const char* nq_last_error(void) { return g_last_error; }

int32_t nq_version(void) { return 410; }

static nq_status check_encode(const nq_params* p, const void* x, nq_dtype x_dtype, int64_t rows,
                              int64_t cols, int64_t ld_x, uint32_t* codes, uint32_t* beta_idx,
                              float* scales, const char* who) {
  if (nq_status s = check_cols(cols, who)) return s;
  if (nq_status s = check_params(p, cols, who)) return s;
  if (x_dtype != NQ_F32 && x_dtype != NQ_F16 && x_dtype != NQ_BF16)
    return fail(NQ_ERR_UNSUPPORTED, "%s: unsupported input dtype %d", who, (int)x_dtype);
  if (rows < 0 || rows >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: rows=%lld outside [0, 2^31)", who, (long long)rows);
  if (ld_x < cols) return fail(NQ_ERR_INVALID_ARG, "%s: ld_x < cols", who);
  if (rows == 0) return NQ_OK;
  if (!x || !codes || !beta_idx || !scales)
    return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  if (!aligned16(x) || (ld_x * (int64_t)dtype_size(x_dtype)) % 16 != 0)
    return fail(NQ_ERR_INVALID_ARG, "%s: x and its row stride must be 16-byte aligned", who);
  return NQ_OK;
}

static nq::EncodeArgs encode_args(const nq_params* p) {
  nq::EncodeArgs a{};
  a.q = p->q;
  a.k = p->k;
  a.rq = (float)(1.0 / p->q);
  a.m2q = nq::magic_2q(p->q);
  a.mq = nq::magic_q(p->q);
  a.decoder = p->decoder;
  a.strategy = p->strategy;
  for (int t = 0; t < 4; ++t) a.beta[t] = (double)beta_mult(p, t) * p->base;
  a.tiles = nullptr;
  a.mtab = mult_table(p);
  return a;
}

nq_status nq_encode(const nq_params* p, const void* x, nq_dtype x_dtype, int64_t rows,
                    int64_t cols, int64_t ld_x, uint32_t* codes, uint32_t* beta_idx,
                    float* scales, void* hip_stream) {
  const char* who = "nq_encode";
  if (nq_status s = check_encode(p, x, x_dtype, rows, cols, ld_x, codes, beta_idx, scales, who))
    return s;
  if (rows == 0) return ok();
  const nq::EncodeArgs a = encode_args(p);
  return hip_status(nq::launch_encode(x, (int)x_dtype, rows, (int)cols, ld_x, a, codes, beta_idx,
                                      scales, (hipStream_t)hip_stream),
                    who);
}

nq_status nq_decode(const nq_params* p, const uint32_t* codes, const uint32_t* beta_idx,
                    const float* scales, int64_t rows, int64_t cols, void* out,
                    nq_dtype out_dtype, int64_t ld_out, void* hip_stream) {
  const char* who = "nq_decode";
  if (nq_status s = check_cols(cols, who)) return s;
  if (nq_status s = check_params(p, cols, who)) return s;
  if (out_dtype != NQ_F32 && out_dtype != NQ_F16 && out_dtype != NQ_BF16)
    return fail(NQ_ERR_UNSUPPORTED, "%s: unsupported output dtype %d", who, (int)out_dtype);
  if (rows < 0 || rows >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: rows=%lld outside [0, 2^31)", who, (long long)rows);
  if (ld_out < cols) return fail(NQ_ERR_INVALID_ARG, "%s: ld_out < cols", who);
  if (rows == 0) return ok();
  if (!codes || !beta_idx || !scales || !out)
    return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  if (!aligned16(out) || (ld_out * (int64_t)dtype_size(out_dtype)) % 16 != 0)
    return fail(NQ_ERR_INVALID_ARG, "%s: out and its row stride must be 16-byte aligned", who);
  nq::DecodeArgs a;
  a.q = p->q;
  a.m2q = nq::magic_2q(p->q);
  a.decoder = p->decoder;
  for (int t = 0; t < 4; ++t) a.half_beta[t] = ((double)beta_mult(p, t) * p->base) * 0.5;
  return hip_status(nq::launch_decode(codes, beta_idx, scales, rows, (int)cols, out,
                                      (int)out_dtype, ld_out, a, (hipStream_t)hip_stream),
                    who);
}

static nq_status check_matmul(const nq_params* pa, const uint32_t* a_codes,
                              const uint32_t* a_beta, const float* a_scales, int64_t M,
                              const nq_params* pw, const uint32_t* w_codes,
                              const uint32_t* w_beta, const float* w_scales, int64_t N,
                              int64_t K, float* c, int64_t ldc, const char* who) {
  if (nq_status s = check_cols(K, who)) return s;
  if (nq_status s = check_params(pa, K, who)) return s;
  if (nq_status s = check_params(pw, K, who)) return s;
  if (M < 0 || M >= kMaxRows || N < 0 || N >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: M, N must be in [0, 2^31)", who);
  if (ldc < N) return fail(NQ_ERR_INVALID_ARG, "%s: ldc < N", who);
  if (M == 0 || N == 0) return NQ_OK;
  if (!a_codes || !a_beta || !a_scales || !w_codes || !w_beta || !w_scales || !c)
    return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  return NQ_OK;
}

// The rotation of rows of `cols` entries inside the encoder: NQ_ERR_UNSUPPORTED unless the
// encoder's one-row-per-workgroup instantiations can hold and rotate them.
static nq_status rotation_args(const nq_params* p, int64_t cols, nq::EncodeArgs& a,
                               const char* who) {
  if (!nq::encode_rotates((int)cols, p->strategy))
    return fail(NQ_ERR_UNSUPPORTED,
                "%s: rotating while coding needs First-beta and cols in {3584, 4096, 7168, 8192, "
                "14336, 16384} (got cols=%lld, strategy=%d); call nq_rotate, then nq_encode",
                who, (long long)cols, p->strategy);
  int pp = 0;
  nq::rotation_split(cols, pp);
  int lp = 0;
  while ((1 << lp) < pp) ++lp;
  a.rot_p = pp;
  a.rot_lp = lp;
  a.rot_s = (float)(1.0 / std::sqrt((double)cols));   // as nq_rotate's scaling
  return NQ_OK;
}

nq_status nq_rotate_encode(const nq_params* p, const void* x, nq_dtype x_dtype, int64_t rows,
                           int64_t cols, int64_t ld_x, uint32_t* codes, uint32_t* beta_idx,
                           float* scales, void* hip_stream) {
  const char* who = "nq_rotate_encode";
  if (nq_status s = check_encode(p, x, x_dtype, rows, cols, ld_x, codes, beta_idx, scales, who))
    return s;
  nq::EncodeArgs a = encode_args(p);
  if (nq_status s = rotation_args(p, cols, a, who)) return s;
  if (rows == 0) return ok();
  return hip_status(nq::launch_encode(x, (int)x_dtype, rows, (int)cols, ld_x, a, codes, beta_idx,
                                      scales, (hipStream_t)hip_stream),
                    who);
}

nq_status nq_rotate(const void* x, nq_dtype x_dtype, int64_t rows, int64_t cols, int64_t ld_x,
                    float* y, int64_t ld_y, void* hip_stream) {
  const char* who = "nq_rotate";
  if (x_dtype != NQ_F32 && x_dtype != NQ_F16 && x_dtype != NQ_BF16)
    return fail(NQ_ERR_UNSUPPORTED, "%s: unsupported input dtype %d", who, (int)x_dtype);
  int p = 0;
  if (cols < 8 || nq::rotation_split(cols, p) == 0)
    return fail(NQ_ERR_UNSUPPORTED, "%s: cols=%lld is not 2^k or 28 * 2^k (2^k >= 8, <= %d)",
                who, (long long)cols, nq::kRotateMaxCols);
  if (rows < 0 || rows >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: rows=%lld outside [0, 2^31)", who, (long long)rows);
  if (ld_x < cols || ld_y < cols) return fail(NQ_ERR_INVALID_ARG, "%s: ld < cols", who);
  if (rows == 0) return ok();
  if (!x || !y) return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  if (!aligned16(x) || (ld_x * (int64_t)dtype_size(x_dtype)) % 16 != 0 || !aligned16(y) ||
      (ld_y * 4) % 16 != 0)
    return fail(NQ_ERR_INVALID_ARG, "%s: rows must be 16-byte aligned", who);
  const char* xb = (const char*)x;
  const char* yb = (const char*)y;
  const int64_t xbytes = ((rows - 1) * ld_x + cols) * (int64_t)dtype_size(x_dtype);
  const int64_t ybytes = ((rows - 1) * ld_y + cols) * 4;
  if (xb < yb + ybytes && yb < xb + xbytes)
    return fail(NQ_ERR_INVALID_ARG, "%s: x and y overlap", who);
  static PerDevice attrs(nq::rotate_set_attributes);
  const hipError_t attr_err = attrs.ensure((hipStream_t)hip_stream);
  if (attr_err != hipSuccess) return hip_status(attr_err, who);
  return hip_status(nq::launch_rotate(x, (int)x_dtype, rows, (int)cols, ld_x, y, ld_y,
                                      (hipStream_t)hip_stream),
                    who);
}

nq_status nq_beta_stats(int32_t q, int32_t decoder, const float* v, int64_t n,
                        const double* betas, int32_t m, double* mse, uint8_t* overload,
                        void* hip_stream) {
  const char* who = "nq_beta_stats";
  if (q < 2 || q > 16) return fail(NQ_ERR_INVALID_ARG, "%s: q=%d outside [2,16]", who, q);
  if (decoder != NQ_DECODER_FULL && decoder != NQ_DECODER_M)
    return fail(NQ_ERR_INVALID_ARG, "%s: decoder=%d is not an nq_decoder", who, decoder);
  if (m < 1 || m > 64) return fail(NQ_ERR_INVALID_ARG, "%s: m=%d outside [1,64]", who, m);
  if (n < 0 || n >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: n=%lld outside [0, 2^31)", who, (long long)n);
  if (!betas) return fail(NQ_ERR_INVALID_ARG, "%s: betas is NULL", who);
  nq::BetaGrid g{};
  g.m = m;
  for (int i = 0; i < m; ++i) {
    if (!std::isfinite(betas[i]) || !(betas[i] > 0.0) || (i > 0 && !(betas[i] > betas[i - 1])))
      return fail(NQ_ERR_INVALID_ARG, "%s: betas must be finite, > 0 and increasing", who);
    g.beta[i] = betas[i];
  }
  if (n == 0) return ok();
  if (!v || !mse || !overload) return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  if (!aligned16(v)) return fail(NQ_ERR_INVALID_ARG, "%s: v must be 16-byte aligned", who);
  return hip_status(nq::launch_beta_stats(v, n, g, q, decoder, mse, overload,
                                          (hipStream_t)hip_stream),
                    who);
}

int64_t nq_beta_dp_workspace_size(int64_t n, int32_t m) {
  if (n < 0 || n >= kMaxRows || m < 1 || m > 64) return -1;
  return (int64_t)nq::beta_dp_workspace(n, m);
}

nq_status nq_beta_dp(const double* mse, const uint8_t* overload, int64_t n, int32_t m,
                     int32_t k, int32_t* chosen, double* loss, void* workspace,
                     int64_t workspace_bytes, void* hip_stream) {
  const char* who = "nq_beta_dp";
  if (m < 1 || m > 64) return fail(NQ_ERR_INVALID_ARG, "%s: m=%d outside [1,64]", who, m);
  if (k < 1 || k > m) return fail(NQ_ERR_INVALID_ARG, "%s: k=%d outside [1, m]", who, k);
  if (n < 0 || n >= kMaxRows)
    return fail(NQ_ERR_INVALID_ARG, "%s: n=%lld outside [0, 2^31)", who, (long long)n);
  if ((n > 0 && (!mse || !overload)) || !chosen || !loss)
    return fail(NQ_ERR_INVALID_ARG, "%s: NULL array pointer", who);
  const int64_t need = nq_beta_dp_workspace_size(n, m);
  if (!workspace || workspace_bytes < need)
    return fail(NQ_ERR_INVALID_ARG, "%s: workspace of %lld bytes needed", who, (long long)need);
  if (((uintptr_t)workspace & 7u) != 0)
    return fail(NQ_ERR_INVALID_ARG, "%s: workspace must be 8-byte aligned", who);
  return hip_status(nq::launch_beta_dp(mse, overload, n, m, k, chosen, loss, workspace,
                                       (hipStream_t)hip_stream),
                    who);
}

int64_t nq_matmul_workspace_size(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 8 || K % 8 || K > kMaxCols) return -1;
  if (M == 0 || N == 0) return 0;
  if (M <= nq::kFusedMaxM) return (int64_t)nq::skinny_workspace(M, K);
  return (int64_t)nq::decode_once_workspace(M, N, K);
}

// Element type of the product's tiles: int8 on request (2q * mult_k <= 127 for both
// operands), else bf16 while every |m X2| <= 256, else fp16 (exact up to 2048).
static nq_status elem_type(const nq_params* pa, const nq_params* pw, bool i8, int& et,
                           const char* who) {
  if (i8 && (tile_bound(pa) > 127 || tile_bound(pw) > 127))
    return fail(NQ_ERR_UNSUPPORTED,
                "%s: the int8 contraction needs 2q * mult_k <= 127 for both operands (k * q <= "
                "63 on the uniform grid; |m X2| must fit int8)", who);
  et = i8 ? nq::ET_I8
          : (tile_bound(pa) <= 256 && tile_bound(pw) <= 256 ? nq::ET_BF16 : nq::ET_F16);
  return NQ_OK;
}

static nq_status check_workspace(int64_t M, int64_t N, int64_t K, void* workspace,
                                 int64_t workspace_bytes, const char* who) {
  const int64_t need = nq_matmul_workspace_size(M, N, K);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(NQ_ERR_INVALID_ARG, "%s: workspace of %lld bytes needed", who, (long long)need);
  if (need > 0 && !aligned16(workspace))
    return fail(NQ_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);
  return NQ_OK;
}

// Padded row length, in blocks, of the activation's tile in the workspace (both paths pad K
// to 128 bytes per row of tiles).
static int tile_blocks(int64_t K, int et) {
  const int64_t eb = et == nq::ET_I8 ? 1 : 2;
  return (int)((K * eb + 127) / 128 * 128 / eb / 8);
}

static hipError_t launch_product(int stages, int et, const nq_params* pa, const nq_params* pw,
                                 const nq::MatmulOperand& A, const nq::MatmulOperand& W,
                                 int64_t K, float* c, int64_t ldc, void* workspace,
                                 hipStream_t st) {
  const float scale = (float)(pa->base * pw->base * 0.25);
  if (A.rows <= nq::kFusedMaxM)
    return nq::launch_matmul_skinny(stages, et, A, W, K, c, ldc, scale, workspace, st);
  static PerDevice attrs(nq::gemm_set_attributes);
  const hipError_t attr_err = attrs.ensure(st);
  if (attr_err != hipSuccess) return attr_err;
  return nq::launch_matmul_decode_once(stages, et, A, W, K, c, ldc, scale, workspace, st);
}

}  // extern "C"

nq_status nq::matmul_stages(int32_t stages, const nq_params* pa, const uint32_t* a_codes,
                            const uint32_t* a_beta, const float* a_scales, int64_t M,
                            const nq_params* pw, const uint32_t* w_codes,
                            const uint32_t* w_beta, const float* w_scales, int64_t N, int64_t K,
                            float* c, int64_t ldc, void* workspace, int64_t workspace_bytes,
                            void* hip_stream, const char* who) {
  if ((stages & ~(NQ_STAGE_DECODE | NQ_STAGE_CONTRACT | NQ_CONTRACT_INT8)) != 0 ||
      (stages & (NQ_STAGE_DECODE | NQ_STAGE_CONTRACT)) == 0)
    return fail(NQ_ERR_INVALID_ARG,
                "%s: stages must hold NQ_STAGE_DECODE and/or NQ_STAGE_CONTRACT, plus optionally "
                "NQ_CONTRACT_INT8", who);
  if (nq_status s = check_matmul(pa, a_codes, a_beta, a_scales, M, pw, w_codes, w_beta,
                                 w_scales, N, K, c, ldc, who))
    return s;
  int et = 0;
  if (nq_status s = elem_type(pa, pw, (stages & NQ_CONTRACT_INT8) != 0, et, who)) return s;
  if (M == 0 || N == 0) return ok();
  if (nq_status s = check_workspace(M, N, K, workspace, workspace_bytes, who)) return s;
  nq::MatmulOperand A{a_codes, a_beta, a_scales, pa->q, nq::magic_2q(pa->q), M, pa->decoder,
                      mult_table(pa)};
  nq::MatmulOperand W{w_codes, w_beta, w_scales, pw->q, nq::magic_2q(pw->q), N, pw->decoder,
                      mult_table(pw)};
  return hip_status(launch_product(stages, et, pa, pw, A, W, K, c, ldc, workspace,
                                   (hipStream_t)hip_stream),
                    who);
}

extern "C" {

nq_status nq_matmul_ex(const nq_params* pa, const uint32_t* a_codes, const uint32_t* a_beta,
                       const float* a_scales, int64_t M, const nq_params* pw,
                       const uint32_t* w_codes, const uint32_t* w_beta, const float* w_scales,
                       int64_t N, int64_t K, float* c, int64_t ldc, void* workspace,
                       int64_t workspace_bytes, void* hip_stream) {
  return nq::matmul_stages(NQ_STAGE_DECODE | NQ_STAGE_CONTRACT, pa, a_codes, a_beta, a_scales, M,
                       pw, w_codes, w_beta, w_scales, N, K, c, ldc, workspace, workspace_bytes,
                       hip_stream, "nq_matmul_ex");
}

nq_status nq_matmul_stages(int32_t stages, const nq_params* pa, const uint32_t* a_codes,
                           const uint32_t* a_beta, const float* a_scales, int64_t M,
                           const nq_params* pw, const uint32_t* w_codes, const uint32_t* w_beta,
                           const float* w_scales, int64_t N, int64_t K, float* c, int64_t ldc,
                           void* workspace, int64_t workspace_bytes, void* hip_stream) {
  return nq::matmul_stages(stages, pa, a_codes, a_beta, a_scales, M, pw, w_codes, w_beta, w_scales,
                       N, K, c, ldc, workspace, workspace_bytes, hip_stream, "nq_matmul_stages");
}

nq_status nq_matmul(const nq_params* pa, const uint32_t* a_codes, const uint32_t* a_beta,
                    const float* a_scales, int64_t M, const nq_params* pw,
                    const uint32_t* w_codes, const uint32_t* w_beta, const float* w_scales,
                    int64_t N, int64_t K, float* c, int64_t ldc, void* hip_stream) {
  const char* who = "nq_matmul";
  if (nq_status s = check_matmul(pa, a_codes, a_beta, a_scales, M, pw, w_codes, w_beta,
                                 w_scales, N, K, c, ldc, who))
    return s;
  int et = 0;
  if (nq_status s = elem_type(pa, pw, false, et, who)) return s;
  if (M == 0 || N == 0) return ok();
  hipStream_t st = (hipStream_t)hip_stream;
  static PerDevice attrs(nq::fused_set_attributes);
  const hipError_t attr_err = attrs.ensure(st);
  if (attr_err != hipSuccess) return hip_status(attr_err, who);
  nq::MatmulOperand A{a_codes, a_beta, a_scales, pa->q, nq::magic_2q(pa->q), M, pa->decoder,
                      mult_table(pa)};
  nq::MatmulOperand W{w_codes, w_beta, w_scales, pw->q, nq::magic_2q(pw->q), N, pw->decoder,
                      mult_table(pw)};
  const float scale = (float)(pa->base * pw->base * 0.25);
  return hip_status(nq::launch_matmul_fused(et, A, W, K, c, ldc, scale, st), who);
}


nq_status nq_encode_matmul(int32_t flags, const nq_params* pa, const void* x, nq_dtype x_dtype,
                           int64_t M, int64_t K, int64_t ld_x, uint32_t* a_codes,
                           uint32_t* a_beta, float* a_scales, const nq_params* pw,
                           const uint32_t* w_codes, const uint32_t* w_beta,
                           const float* w_scales, int64_t N, float* c, int64_t ldc,
                           void* workspace, int64_t workspace_bytes, void* hip_stream) {
  const char* who = "nq_encode_matmul";
  if ((flags & ~(NQ_CONTRACT_INT8 | NQ_ROTATE_A)) != 0)
    return fail(NQ_ERR_INVALID_ARG, "%s: flags may only hold NQ_CONTRACT_INT8, NQ_ROTATE_A", who);
  if (nq_status s = check_encode(pa, x, x_dtype, M, K, ld_x, a_codes, a_beta, a_scales, who))
    return s;
  nq::EncodeArgs a = encode_args(pa);
  if (flags & NQ_ROTATE_A)
    if (nq_status s = rotation_args(pa, K, a, who)) return s;
  if (nq_status s = check_matmul(pa, a_codes, a_beta, a_scales, M, pw, w_codes, w_beta,
                                 w_scales, N, K, c, ldc, who))
    return s;
  int et = 0;
  if (nq_status s = elem_type(pa, pw, (flags & NQ_CONTRACT_INT8) != 0, et, who)) return s;
  if (M == 0 || N == 0) return ok();
  if (nq_status s = check_workspace(M, N, K, workspace, workspace_bytes, who)) return s;
  hipStream_t st = (hipStream_t)hip_stream;
  nq::MatmulOperand A{a_codes, a_beta, a_scales, pa->q, nq::magic_2q(pa->q), M, pa->decoder,
                      mult_table(pa)};
  nq::MatmulOperand W{w_codes, w_beta, w_scales, pw->q, nq::magic_2q(pw->q), N, pw->decoder,
                      mult_table(pw)};
  // 1. encode A; the encoder also writes A's decoded tiles into the workspace and, on the
  //    decode-once path where its instantiation allows, W's tile decode rides in the same
  //    launch (workgroups after the encoder's, which fill the encoder's tail)
  const int nbp = tile_blocks(K, et);
  const int64_t rows_p = M <= nq::kFusedMaxM ? (M + 15) / 16 * 16 : (M + 255) / 256 * 256;
  a.tiles = workspace;
  a.tile_et = et;
  a.nb_p = nbp;
  int stages = nq::kStageDecodeW | NQ_STAGE_CONTRACT;
  if (M > nq::kFusedMaxM && nq::encode_carries_task((int)K, pa->strategy)) {
    int64_t w_offset, np;
    int wnbp;
    nq::decode_once_layout(et, M, N, K, w_offset, np, wnbp);
    a.task = nq::tile_task(W, (int)(K / 8), np, wnbp,
                           static_cast<unsigned char*>(workspace) + w_offset);
    stages = NQ_STAGE_CONTRACT;
  }
  hipError_t e = nq::launch_encode(x, (int)x_dtype, M, (int)K, ld_x, a, a_codes, a_beta,
                                   a_scales, st);
  if (e == hipSuccess) e = nq::launch_tiles_pad(et, workspace, M, (int)(K / 8), rows_p, nbp, st);
  if (e != hipSuccess) return hip_status(e, who);
  // 2. decode W (unless the encoder's launch did) and contract
  return hip_status(launch_product(stages, et, pa, pw, A, W, K, c, ldc, workspace, st), who);
}

}  // extern "C"

/*
 * nestquant.h -- C ABI of the MI355X NestQuant coded-GEMM library (libnestquant.so).
 *
 * NestQuant (Savkin, Porat, Ordentlich, Polyanskiy, arXiv 2502.09720) quantizes every row
 * of a matrix with a union of k scaled Voronoi codes of the Gosset lattice E8 and
 * computes matrix products from the codes.  This library implements, for one AMD
 * Instinct MI355X (gfx950):
 *
 *   nq_encode  -- Sec. 4.2, Alg. 3 (row quantizer) with the First-beta strategy of App. F,
 *                 built on Alg. 1 (Voronoi encode) and App. C, Alg. 5 (nearest E8 point);
 *   nq_decode  -- Alg. 2 (Voronoi decode) scaled back by beta and the row scale;
 *   nq_matmul  -- C = A_hat * W_hat^T from two coded operands, i.e. Alg. 4 (dot product of
 *                 coded vectors) for every pair of rows, as one dense contraction.
 *
 * Storage of a coded matrix with `rows` rows of `cols` entries (cols % 8 == 0):
 *   codes    uint32[rows][cols/8]           block j of row i: code c_l (0 <= c_l < q) of
 *                                           entry 8j+l in bits 4l..4l+3 (App. E packs the
 *                                           eight codes of a block into one 32-bit word);
 *   beta_idx uint32[rows][ceil(cols/128)]   two bits per block: (t - 1) of block j in bits
 *                                           2*(j%16) of word j/16 (App. E: 2-bit indices
 *                                           into a dictionary of four betas);
 *   scales   float[rows]                    r = ||row||_2 / sqrt(cols), the fp32 number
 *                                           nearest to the exact value (Alg. 3's s/sqrt(n)).
 * The value coded for entry 8j+l is  r * beta_t * p_l  with beta_t = t * base and p the
 * decoded E8 point; beta_t = t * base for t = 1..k is the beta dictionary (App. F).
 *
 * Conventions for every call:
 *   - all array pointers are device pointers, owned by the caller; the library keeps no
 *     per-call state and allocates no memory: calls that need scratch memory take a
 *     caller-owned workspace and have a size query (nq_matmul_ex, nq_beta_dp);
 *   - calls are asynchronous on `hip_stream` (a hipStream_t; NULL = the null stream) and
 *     may be issued from several host threads;
 *   - arguments are checked on the host before anything is launched: on any error the
 *     call returns the status, launches nothing and writes nothing; nq_last_error() then
 *     describes the failure (per host thread);
 *   - rows == 0 (or M == 0 / N == 0) is a no-op returning NQ_OK.
 */
#ifndef NESTQUANT_H
#define NESTQUANT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NQ_OK = 0,
  NQ_ERR_INVALID_ARG = 1,  /* a size, stride, pointer or parameter is out of range   */
  NQ_ERR_UNSUPPORTED = 2,  /* valid in principle but not implemented (e.g. dtype)    */
  NQ_ERR_HIP = 3,          /* the HIP runtime reported an error at launch            */
  NQ_STATUS_MAX_ENUM = 0x7FFFFFFF
} nq_status;

/* Every enum of this ABI has a MAX_ENUM member, so that it is 32 bits wide and any int32
 * value a caller passes is a value of the type (invalid ones are then rejected by value). */
typedef enum { NQ_F32 = 0, NQ_F16 = 1, NQ_BF16 = 2, NQ_DTYPE_MAX_ENUM = 0x7FFFFFFF } nq_dtype;

/* Decoder of the code (part of its definition: the encoder's overload test uses it).
 *   NQ_DECODER_FULL  Alg. 2 with the Gosset oracle of Alg. 5 (App. C);
 *   NQ_DECODER_M     NestQuantM (App. D): the oracle's parity fixes at the first coordinate
 *                    (no argmin / argmax); the encoder is unchanged except that a point
 *                    counts as overloaded when this decoder does not reproduce it. */
typedef enum { NQ_DECODER_FULL = 0, NQ_DECODER_M = 1, NQ_DECODER_MAX_ENUM = 0x7FFFFFFF } nq_decoder;

/* How the encoder picks one of the k betas for a block (App. F).  Both give the same code
 * format; decoding and the matrix product do not look at it.
 *   NQ_FIRST_BETA  the smallest beta that does not overload (t = k if all do);
 *   NQ_OPT_BETA    every beta is tried and the one whose reconstruction
 *                  beta_t * X2_t / 2 is nearest to the normalized block x / r is kept: the
 *                  error is sum over l = 0..7, in that order, of d_l^2 with
 *                  d_l = fl64(fl64(beta_t * X2_t,l) / 2 - fl64(x_l / r)), every step
 *                  rounded in fp64, and the first t with the least error wins. */
typedef enum { NQ_FIRST_BETA = 0, NQ_OPT_BETA = 1, NQ_STRATEGY_MAX_ENUM = 0x7FFFFFFF } nq_strategy;

/* Quantizer parameters (Sec. 4.2, App. F):
 *   q        nesting ratio, 2 <= q <= 16 (codes are nibbles);
 *   k        number of betas, 1 <= k <= 4 (2-bit beta indices);
 *   base     beta_t = mult_t * base for t = 1..k; finite, > 0, and large enough that
 *            sqrt(cols) / base < 2^21 (bounds the lattice input |y| <= sqrt(cols) / base).
 *            The paper's grid "k betas uniform on [0, 10] / q" is base = 10 / (k q) with
 *            mult_t = t;
 *   decoder  an nq_decoder value (0 = Alg. 2 / Alg. 5);
 *   strategy an nq_strategy value (0 = First-beta); used by nq_encode only;
 *   mult     the integer multiples of base: all zero for (1, 2, 3, 4) (the uniform grid), or
 *            1 <= mult[0] < ... < mult[k-1] <= 64 with mult[k..3] = 0, e.g. a set chosen by
 *            the dynamic program of App. F from the grid (1/2) {1, ..., 50} / q, which is
 *            base = 1 / (2q) with multiples 1..50.  Each beta is fl64(mult_t * base).
 * Codes made with one decoder must be decoded and multiplied with the same one, and with
 * the same base and mult. */
typedef struct {
  int32_t q;
  int32_t k;
  double base;
  int32_t decoder;
  int32_t strategy;
  int32_t mult[4];
} nq_params;

/* Alg. 3 with the beta strategy p->strategy (App. F) on each row of x.
 *   x        device, rows x cols of dtype x_dtype (NQ_F32, NQ_F16 or NQ_BF16), row i at
 *            x + i*ld_x elements; ld_x >= cols; cols % 8 == 0, 8 <= cols <= 65536.
 *   codes    device, nq_codes_words(rows, cols) uint32 (output);
 *   beta_idx device, nq_beta_words(rows, cols) uint32 (output);
 *   scales   device, rows floats (output).
 * Per row: r = RMS; for every 8-block, for t = 1..k the block y = fl32(x * c_t) with
 * c_t = fl32(1 / fl64(r * beta_t)) is rounded to the nearest E8 point (Alg. 5;
 * ties: exact halves round down, lowest index on argmin/argmax ties, equal D8 / D8+1/2
 * distances pick D8+1/2).  First-beta keeps the first t whose point survives
 * decode(encode(.)) (no overload, Sec. 4.1), else t = k; Opt-beta keeps the t of least
 * reconstruction error (nq_strategy).  A zero row gives r = 0, codes 0, index 0.
 * Non-finite inputs give unspecified (but in-range) codes. */
nq_status nq_encode(const nq_params* p, const void* x, nq_dtype x_dtype, int64_t rows,
                    int64_t cols, int64_t ld_x, uint32_t* codes, uint32_t* beta_idx,
                    float* scales, void* hip_stream);

/* Alg. 2 and the inverse scaling: out[i][8j+l] = r_i * beta_t * X2_l / 2 where X2
 * is the decoded point of block j in 2E8 units (App. E).  out is rows x cols of out_dtype,
 * row i at out + i*ld_out elements, ld_out >= cols.  Each value is the fp64 product rounded
 * once to fp32 (and, for NQ_F16 / NQ_BF16, from there to the 16-bit type). */
nq_status nq_decode(const nq_params* p, const uint32_t* codes, const uint32_t* beta_idx,
                    const float* scales, int64_t rows, int64_t cols, void* out,
                    nq_dtype out_dtype, int64_t ld_out, void* hip_stream);

/* C = A_hat * W_hat^T (Alg. 4 for every row pair), fp32 output, with no workspace.
 *   A: M x K coded with parameters pa; W: N x K coded with parameters pw (q, k, base and
 *   mult may differ between the operands; K must be the same);  K % 8 == 0, K <= 65536.
 *   c: device, M x N floats, row i at c + i*ldc, ldc >= N.
 * C_ij = r_Ai r_Wj base_A base_W / 4 * sum_blocks <m_A X2_A, m_W X2_W> (m = mult_t of the
 * block's beta); the integer tiles m*X2 are contracted with fp32 accumulation on bf16
 * matrix cores, exact in bf16 when 2q * mult_k <= 256 for both operands (always so for the
 * uniform grid), else on fp16 matrix cores (exact up to 2048, every allowed mult).
 * Each workgroup decodes (Alg. 2) the code words of its own rows of A and W into on-chip
 * memory and contracts them there, so the call needs and allocates no memory; a block of A is
 * decoded once per 128 columns of C (64 for M <= 64) and a block of W once per 256 rows of C
 * (64 for M <= 64).  nq_matmul_ex computes the same product decoding every block exactly
 * once into a caller's workspace, which is faster once M is in the hundreds; for M > 64 the
 * two sum in the same order and agree bit for bit. */
nq_status nq_matmul(const nq_params* pa, const uint32_t* a_codes, const uint32_t* a_beta,
                    const float* a_scales, int64_t M, const nq_params* pw,
                    const uint32_t* w_codes, const uint32_t* w_beta, const float* w_scales,
                    int64_t N, int64_t K, float* c, int64_t ldc, void* hip_stream);

/* nq_matmul with a caller-owned device workspace (16-byte aligned, at least
 * nq_matmul_workspace_size(M, N, K) bytes): every block of both operands is decoded exactly
 * once (Alg. 2) into integer tiles m*X2 in the workspace (for M <= 64 only A's; W is then
 * decoded straight into matrix-core operands), then contracted.  Same product as nq_matmul
 * (for M <= 64 the fp32 sums are taken in another order).  With M <= 2 (and A's tile within
 * 48 KiB) the product kernel decodes A itself and the workspace is unused; there, when
 * every sum fits 32 bits (8 * ceil(K / 64) * 8 * (2 q_A)(2 q_W) * max mult_A * max mult_W
 * < 2^31: always at q = 16 with multiples up to 4), each output's sum of
 * <m_A X2_A, m_W X2_W> is exact in int32 (int8 dot products, no matrix cores) and rounded
 * once to fp32.  The workspace is used as scratch until the call's kernels finish on
 * hip_stream. */
nq_status nq_matmul_ex(const nq_params* pa, const uint32_t* a_codes, const uint32_t* a_beta,
                       const float* a_scales, int64_t M, const nq_params* pw,
                       const uint32_t* w_codes, const uint32_t* w_beta, const float* w_scales,
                       int64_t N, int64_t K, float* c, int64_t ldc, void* workspace,
                       int64_t workspace_bytes, void* hip_stream);

/* Bytes of the library's static device scratch used by nq_matmul_static (64 MiB per device). */
#define NQ_STATIC_SCRATCH_BYTES (64u << 20)

/* nq_matmul_ex for callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The workspace is the library's own
 * static device array of NQ_STATIC_SCRATCH_BYTES, which every device the library runs on holds
 * until the process ends; the call allocates nothing (no hipMalloc, no allocating library
 * routine).  Same arguments, checks and results (bit for bit) as nq_matmul_ex without the
 * workspace arguments.  A product whose nq_matmul_workspace_size(M, N, K) exceeds
 * NQ_STATIC_SCRATCH_BYTES is rejected with NQ_ERR_UNSUPPORTED before anything is launched
 * (every product with M <= 64 fits, and so does 2048 x 4096 x 4096).  All calls on one device
 * share its array: calls whose kernels overlap on a device (other streams, other host threads)
 * race and must be serialized by the caller; consecutive calls on one stream are safe. */
nq_status nq_matmul_static(const nq_params* pa, const uint32_t* a_codes, const uint32_t* a_beta,
                           const float* a_scales, int64_t M, const nq_params* pw,
                           const uint32_t* w_codes, const uint32_t* w_beta,
                           const float* w_scales, int64_t N, int64_t K, float* c, int64_t ldc,
                           void* hip_stream);

/* The two stages of nq_matmul_ex, for callers that time or schedule them separately, and
 * the exact int8 contraction.  stages is a bit mask:
 *   NQ_STAGE_DECODE    decodes the operands into the workspace (every block of A and, for
 *                      M > 64, of W, as m*X2);
 *   NQ_STAGE_CONTRACT  computes C from the workspace (for M <= 64 it also decodes W, straight
 *                      into matrix-core operands);
 *   NQ_CONTRACT_INT8   stores m*X2 as int8 and contracts on int8 matrix cores with int32
 *                      accumulation instead of bf16 / fp32.  Every inner product
 *                      sum <m_A X2_A, m_W X2_W> (Alg. 4 without its scale) is then exact, and
 *                      C = fp32(sum) * r_A * r_W * base_A * base_W / 4.  It requires
 *                      2q * mult_k <= 127 for both operands (with the uniform grid: k * q <= 63;
 *                      |m X2| <= 2q m must fit int8), else NQ_ERR_UNSUPPORTED.  Both stages
 *                      of one product must agree on it.
 * A DECODE call followed by a CONTRACT call with the same arguments on the same stream is
 * exactly the call with both bits; DECODE | CONTRACT is nq_matmul_ex.  The workspace must
 * not change in between.  Arguments are validated as in nq_matmul_ex; any other bit, or no
 * stage bit, is NQ_ERR_INVALID_ARG.  The workspace size is nq_matmul_workspace_size either
 * way. */
enum { NQ_STAGE_DECODE = 1, NQ_STAGE_CONTRACT = 2, NQ_CONTRACT_INT8 = 4 };

/* Flag of nq_encode_matmul: rotate the activation's rows before coding them (as
 * nq_rotate_encode; W must then have been coded from rotated rows, W U, so that
 * (A U)(W U)^T = A W^T). */
enum { NQ_ROTATE_A = 8 };
nq_status nq_matmul_stages(int32_t stages, const nq_params* pa, const uint32_t* a_codes,
                           const uint32_t* a_beta, const float* a_scales, int64_t M,
                           const nq_params* pw, const uint32_t* w_codes, const uint32_t* w_beta,
                           const float* w_scales, int64_t N, int64_t K, float* c, int64_t ldc,
                           void* workspace, int64_t workspace_bytes, void* hip_stream);

/* Online rotation of rows before quantization (Sec. 5, "LLM quantization"): y = x U for
 * every row, with U = H_n / sqrt(n) (Sylvester's Hadamard matrix) when cols = n = 2^k, and
 * U = (H_28 kron H_{2^k}) / sqrt(n) when n = 28 * 2^k (Llama-3's 14336 and 28672), H_28 from
 * Paley's second construction at q = 13.  Since U is orthogonal, A W^T = (A U)(W U)^T: the
 * rotation spreads outlier channels before nq_encode.
 *   x    device, rows x cols of x_dtype, row i at x + i * ld_x (16-byte aligned rows);
 *   y    device fp32 rows x cols, row i at y + i * ld_y (16-byte aligned rows); may not
 *        overlap x.
 * Supported: cols = 2^k or 28 * 2^k with 2^k >= 8 and cols <= 32768, else
 * NQ_ERR_UNSUPPORTED.  Arithmetic: fp32 fast Walsh-Hadamard transform (stages h = 1, 2, 4, ...
 * along each length-2^k segment); then for 28 * 2^k, output segment a is the sum over
 * i = 0..27, in increasing i, of H_28[i][a] X_i (X_i the i-th segment, each term an exact
 * +-X_i, one fp32 rounding per addition); then one multiplication by fl32(1 / sqrt(n)).
 * rows == 0 is a no-op. */
nq_status nq_rotate(const void* x, nq_dtype x_dtype, int64_t rows, int64_t cols, int64_t ld_x,
                    float* y, int64_t ld_y, void* hip_stream);

/* nq_rotate followed by nq_encode in one pass (Sec. 5: the rotation in front of the
 * quantizer): every row of x is rotated in on-chip memory with nq_rotate's arithmetic and
 * coded from there, so the fp32 rotated rows never go to memory.  Codes, beta indices and
 * scales equal those of nq_encode on nq_rotate's output, bit for bit.
 *   p, x, x_dtype, rows, cols, ld_x, codes, beta_idx, scales: as nq_encode.
 * Supported: First-beta, and cols = 3584, 4096, 7168, 8192, 14336 or 16384 (widths nq_rotate
 * supports with 257..2048 blocks per row); else NQ_ERR_UNSUPPORTED (call nq_rotate, then
 * nq_encode).  Validation as nq_encode; rows == 0 is a no-op. */
nq_status nq_rotate_encode(const nq_params* p, const void* x, nq_dtype x_dtype, int64_t rows,
                           int64_t cols, int64_t ld_x, uint32_t* codes, uint32_t* beta_idx,
                           float* scales, void* hip_stream);

/* Workspace bytes nq_matmul_ex needs for an M x N x K product (0 when M or N is 0; -1 for
 * an invalid K). */
int64_t nq_matmul_workspace_size(int64_t M, int64_t N, int64_t K);

/* The whole hot path in one call: Alg. 3 on the rows of the activation x (as nq_encode,
 * writing A's codes, beta indices and scales), then C = A_hat * W_hat^T from the codes (as
 * nq_matmul_ex).  The encoder also writes A's decoded tiles m * X2 (Alg. 2 of the codes it
 * has just chosen; the lattice point itself wherever it passed the overload test) straight
 * into the product's workspace, so A is never decoded in a separate pass.  W is decoded as in
 * nq_matmul_ex; for M > 64 and First-beta rows of 2056..16384 entries that decode runs in
 * the encoder's launch, after its workgroups.  Results are those of nq_encode followed by
 * nq_matmul_ex (with
 * NQ_CONTRACT_INT8 in flags, of nq_matmul_stages with that flag; with NQ_ROTATE_A, of
 * nq_rotate_encode in place of nq_encode).
 *   flags    0, or NQ_CONTRACT_INT8 and / or NQ_ROTATE_A (the widths and strategy of
 *            nq_rotate_encode, else NQ_ERR_UNSUPPORTED);
 *   x, x_dtype, M (rows), K (cols), ld_x, a_codes, a_beta, a_scales: as nq_encode with pa;
 *   pw, w_codes, w_beta, w_scales, N, c, ldc: as nq_matmul_ex;
 *   workspace: device, 16-byte aligned, at least nq_matmul_workspace_size(M, N, K) bytes.
 * Validation as nq_encode and nq_matmul_ex; nothing is launched on error. */
nq_status nq_encode_matmul(int32_t flags, const nq_params* pa, const void* x, nq_dtype x_dtype,
                           int64_t M, int64_t K, int64_t ld_x, uint32_t* a_codes,
                           uint32_t* a_beta, float* a_scales, const nq_params* pw,
                           const uint32_t* w_codes, const uint32_t* w_beta,
                           const float* w_scales, int64_t N, float* c, int64_t ldc,
                           void* workspace, int64_t workspace_bytes, void* hip_stream);

/* Statistics for choosing the beta set (App. F): for n sample 8-vectors v (normalized as
 * Alg. 3 normalizes rows, i.e. x / r) and m candidate betas, the squared error of coding
 * v_p at beta_i and whether that coding overloads.
 *   q, decoder  the code: 2 <= q <= 16 and an nq_decoder value;
 *   v        device, n x 8 floats, 16-byte aligned (input);
 *   betas    host, m doubles, finite, > 0 and strictly increasing, 1 <= m <= 64;
 *   mse      device, n x m doubles, row p at mse + p*m (output);
 *   overload device, n x m bytes, 1 where the coding overloads, else 0 (output).
 * Per pair: y = fl32(v_p * fl32(1 / beta_i)); P = the nearest E8 point (Alg. 5 with
 * nq_encode's tie rules); X2 = decode(encode(P)) with the decoder (Alg. 1, 2); overload is
 * X2 != P (Sec. 4.1); mse = sum over l = 0..7, in that order, of d_l^2 with
 * d_l = fl64(fl64(beta_i * X2_l) / 2 - v_l), every step rounded in fp64.  Samples with
 * |v| / beta_1 >= 2^21 or non-finite entries give unspecified values.  n = 0 is a no-op;
 * n < 2^31. */
nq_status nq_beta_stats(int32_t q, int32_t decoder, const float* v, int64_t n,
                        const double* betas, int32_t m, double* mse, uint8_t* overload,
                        void* hip_stream);

/* Alg. 6 (App. F): the k of the m grid betas that minimize the First-beta error of the n
 * samples under the DP's model, from nq_beta_stats' outputs (device mse and overload, n x m).
 *   1 <= k <= m <= 64; n < 2^31;
 *   chosen    device, k int32 (output): the indices into the grid, increasing, or all -1 if
 *             every grid beta overloads some sample;
 *   loss      device, one double (output): the minimized total squared error (+inf with -1s);
 *   workspace device, 8-byte aligned, at least nq_beta_dp_workspace_size(n, m) bytes of
 *             scratch, used until the call's kernels finish on hip_stream.
 * dp[i][j] is the least total error of the samples that do not overload at beta_i, coded
 * with beta_i and j - 1 smaller betas under First-beta; the step from the next smaller chosen
 * beta s adds the errors at beta_i of the samples that overload at beta_s but not at beta_i
 * (s = 0: a virtual beta at which every sample overloads).  The answer is the least dp[i][k]
 * over the betas at which no sample overloads.  Every cost is an fp64 sum over the samples
 * in a fixed 64-ary tree (consecutive groups of 64 terms added in order, then groups of 64
 * of those sums, and so on), so each computed cost and dp value is within (63 d + k) 2^-53
 * of its exact value, relatively (d = ceil(log64 n)); ties go to the smallest index. */
nq_status nq_beta_dp(const double* mse, const uint8_t* overload, int64_t n, int32_t m,
                     int32_t k, int32_t* chosen, double* loss, void* workspace,
                     int64_t workspace_bytes, void* hip_stream);

/* Scratch bytes nq_beta_dp needs for n samples and m betas (about (n / 4096 + 1)
 * (m (m + 1) / 2 + m) doubles; -1 for an invalid n or m). */
int64_t nq_beta_dp_workspace_size(int64_t n, int32_t m);

/* Sizes, in 32-bit words, of the code and beta-index arrays of a rows x cols coded matrix
 * (-1 if rows < 0 or cols is not a positive multiple of 8): one word per 8-block, the eight
 * 4-bit codes of App. E's packing (rows * cols / 8), and one word per 16 blocks of 2-bit
 * beta indices (App. E indexes a dictionary of at most four betas; rows * ceil(cols / 128)).
 * Every coded matrix of the library is stored in arrays of exactly these sizes. */
int64_t nq_codes_words(int64_t rows, int64_t cols);
int64_t nq_beta_words(int64_t rows, int64_t cols);

/* Static description of a status code (the error reporting of this ABI; no paper passage). */
const char* nq_status_string(nq_status s);

/* Message describing the last failed call on this host thread ("" if none). */
const char* nq_last_error(void);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int32_t nq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NESTQUANT_H */

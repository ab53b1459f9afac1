// Host-only checks of the C ABI layer (nq_api.cpp with the launch helpers of nq_host.cpp),
// built with a plain host compiler under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_abi_host.py.  The kernels and the HIP runtime are replaced by stubs that record
// every launch and return an error on request, so that no GPU is needed:
//
//   * every rejected call launches nothing and reports why (nq_last_error, per thread);
//   * a launch that fails surfaces as NQ_ERR_HIP, as does a failing device query;
//   * valid calls reach the launcher the contract names (nq_matmul the in-tile decode with no
//     workspace, nq_matmul_ex the decode-once or skinny path), with the arguments the
//     contract derives (scale, element type, tile padding).
//
// Exit status 0 when every check passes; each failure prints its line.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "nestquant.h"
#include "nq_kernels.hpp"

// ---- stub HIP runtime: the only runtime functions the ABI layer calls -------------------
static hipError_t g_query = hipSuccess;   // returned by the device queries
extern "C" {
hipError_t hipStreamGetDevice(hipStream_t, hipDevice_t* dev) {
  *dev = 0;
  return g_query;
}
hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return g_query;
}
hipError_t hipSetDevice(int) { return g_query; }
const char* hipGetErrorString(hipError_t e) {
  return e == hipSuccess ? "hipSuccess" : "stub HIP error";
}
}

// ---- stub launchers ----------------------------------------------------------------------
static std::vector<std::string> g_calls;       // launcher names, in call order
static hipError_t g_launch = hipSuccess;       // returned by every launcher
static int g_last_et = -1, g_last_stages = -1;
static float g_last_scale = 0.0f;

namespace nq {
static hipError_t rec(const char* name) {
  g_calls.push_back(name);
  return g_launch;
}
hipError_t launch_encode(const void*, int, int64_t, int, int64_t, const EncodeArgs& a,
                         uint32_t*, uint32_t*, float*, hipStream_t) {
  g_last_stages = a.task.wgs;
  return rec(a.rot_p ? "encode_rotated" : (a.tiles ? "encode_tiles" : "encode"));
}
hipError_t launch_decode(const uint32_t*, const uint32_t*, const float*, int64_t, int, void*,
                         int, int64_t, const DecodeArgs&, hipStream_t) {
  return rec("decode");
}
hipError_t launch_tiles_pad(int, void*, int64_t, int, int64_t, int, hipStream_t) {
  return rec("tiles_pad");
}
hipError_t launch_matmul_skinny(int stages, int et, const MatmulOperand&, const MatmulOperand&,
                                int64_t, float*, int64_t, float scale, void*, hipStream_t) {
  g_last_et = et;
  g_last_stages = stages;
  g_last_scale = scale;
  return rec("skinny");
}
hipError_t launch_matmul_decode_once(int stages, int et, const MatmulOperand&,
                                     const MatmulOperand&, int64_t, float*, int64_t, float scale,
                                     void*, hipStream_t) {
  g_last_et = et;
  g_last_stages = stages;
  g_last_scale = scale;
  return rec("decode_once");
}
hipError_t launch_matmul_fused(int et, const MatmulOperand&, const MatmulOperand&, int64_t,
                               float*, int64_t, float scale, hipStream_t) {
  g_last_et = et;
  g_last_scale = scale;
  return rec("fused");
}
hipError_t gemm_set_attributes() { return rec("gemm_attributes"); }
hipError_t fused_set_attributes() { return rec("fused_attributes"); }
hipError_t rotate_set_attributes() { return rec("rotate_attributes"); }
hipError_t launch_rotate(const void*, int, int64_t, int, int64_t, float*, int64_t, hipStream_t) {
  return rec("rotate");
}
hipError_t launch_beta_stats(const float*, int64_t, const BetaGrid&, int, int, double*, uint8_t*,
                             hipStream_t) {
  return rec("beta_stats");
}
hipError_t launch_beta_dp(const double*, const uint8_t*, int64_t, int, int, int32_t*, double*,
                          void*, hipStream_t) {
  return rec("beta_dp");
}
}  // namespace nq

// ---- checks ------------------------------------------------------------------------------
static int g_fail = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #cond);    \
      ++g_fail;                                                       \
    }                                                                 \
  } while (0)

static void* const DEV = reinterpret_cast<void*>(0x10000);     // never dereferenced
static uint32_t* const U = static_cast<uint32_t*>(DEV);
static float* const F = static_cast<float*>(DEV);

static nq_params params(int q = 14, int k = 4) {
  nq_params p{};
  p.q = q;
  p.k = k;
  p.base = 10.0 / (k * q);
  return p;
}

static void reset() {
  g_calls.clear();
  g_launch = hipSuccess;
  g_query = hipSuccess;
  g_last_et = g_last_stages = -1;
  g_last_scale = 0.0f;
}

static bool mentions(const char* who) { return std::strstr(nq_last_error(), who) != nullptr; }

static void encode_and_decode() {
  nq_params p = params();
  reset();
  CHECK(nq_encode(&p, DEV, NQ_BF16, 4, 64, 64, U, U, F, nullptr) == NQ_OK);
  CHECK(g_calls.size() == 1 && g_calls[0] == "encode");
  CHECK(std::strcmp(nq_last_error(), "") == 0);

  // a failing launch is NQ_ERR_HIP, with the runtime's message
  reset();
  g_launch = hipErrorLaunchFailure;
  CHECK(nq_encode(&p, DEV, NQ_BF16, 4, 64, 64, U, U, F, nullptr) == NQ_ERR_HIP);
  CHECK(mentions("nq_encode") && mentions("stub HIP error"));
  reset();
  g_launch = hipErrorLaunchFailure;
  CHECK(nq_decode(&p, U, U, F, 4, 64, DEV, NQ_F16, 64, nullptr) == NQ_ERR_HIP);

  // rejected calls launch nothing
  struct Bad {
    int q, k;
    nq_dtype dt;
    int64_t rows, cols, ld;
    void* x;
  } bad[] = {
      {1, 4, NQ_BF16, 4, 64, 64, DEV},   {17, 4, NQ_BF16, 4, 64, 64, DEV},
      {14, 0, NQ_BF16, 4, 64, 64, DEV},  {14, 5, NQ_BF16, 4, 64, 64, DEV},
      {14, 4, NQ_BF16, 4, 60, 64, DEV},  {14, 4, NQ_BF16, 4, 64, 60, DEV},
      {14, 4, NQ_BF16, -1, 64, 64, DEV}, {14, 4, (nq_dtype)7, 4, 64, 64, DEV},
      {14, 4, NQ_BF16, 4, 64, 64, nullptr},
      {14, 4, NQ_BF16, 4, 64, 64, static_cast<char*>(DEV) + 2},
      {14, 4, NQ_BF16, 4, 64, 68, DEV},  {14, 4, NQ_F32, 4, 65544, 65544, DEV},
  };
  for (const Bad& b : bad) {
    reset();
    nq_params pb = params(b.q, b.k);
    const nq_status s = nq_encode(&pb, b.x, b.dt, b.rows, b.cols, b.ld, U, U, F, nullptr);
    CHECK(s == NQ_ERR_INVALID_ARG || s == NQ_ERR_UNSUPPORTED);
    CHECK(g_calls.empty());
    CHECK(mentions("nq_encode"));
  }
  nq_params pm = params();
  pm.mult[0] = 3;   // mult must be all zero or k increasing values
  reset();
  CHECK(nq_encode(&pm, DEV, NQ_BF16, 4, 64, 64, U, U, F, nullptr) == NQ_ERR_INVALID_ARG);
  CHECK(g_calls.empty());
  nq_params pz = params();
  pz.base = std::nan("");
  CHECK(nq_decode(&pz, U, U, F, 4, 64, DEV, NQ_F16, 64, nullptr) == NQ_ERR_INVALID_ARG);
  CHECK(g_calls.empty());
  // rows == 0 is a no-op that launches nothing, even with NULL pointers
  CHECK(nq_encode(&p, nullptr, NQ_BF16, 0, 64, 64, nullptr, nullptr, nullptr, nullptr) == NQ_OK);
  CHECK(g_calls.empty());
}

static void matmul_paths() {
  nq_params pa = params(), pw = params(7, 4);
  // nq_matmul: the in-tile decode, nothing else, after the per-device attributes
  reset();
  CHECK(nq_matmul(&pa, U, U, F, 300, &pw, U, U, F, 500, 256, F, 500, nullptr) == NQ_OK);
  CHECK(g_calls.size() == 2 && g_calls[0] == "fused_attributes" && g_calls[1] == "fused");
  CHECK(g_last_et == nq::ET_BF16);
  CHECK(g_last_scale == (float)(pa.base * pw.base * 0.25));
  // attributes are set once per device
  reset();
  CHECK(nq_matmul(&pa, U, U, F, 3, &pw, U, U, F, 5, 256, F, 5, nullptr) == NQ_OK);
  CHECK(g_calls.size() == 1 && g_calls[0] == "fused");
  // multiples beyond bf16's exact integers: fp16 tiles
  nq_params pf = params(14, 2);
  pf.base = 1.0 / 28.0;
  pf.mult[0] = 9;
  pf.mult[1] = 16;
  reset();
  CHECK(nq_matmul(&pf, U, U, F, 3, &pw, U, U, F, 5, 256, F, 5, nullptr) == NQ_OK);
  CHECK(g_last_et == nq::ET_F16);
  // a failing device query or launch is NQ_ERR_HIP
  reset();
  g_launch = hipErrorLaunchFailure;
  CHECK(nq_matmul(&pa, U, U, F, 3, &pw, U, U, F, 5, 256, F, 5, nullptr) == NQ_ERR_HIP);
  CHECK(mentions("nq_matmul"));

  // nq_matmul_ex: skinny for M <= 64, decode-once above, with the size query's workspace
  const int64_t ws_small = nq_matmul_workspace_size(64, 500, 256);
  const int64_t ws_big = nq_matmul_workspace_size(65, 500, 256);
  CHECK(ws_small == 64 * 256 * 2);
  CHECK(ws_big == (256 + 512) * 256 * 2);
  reset();
  CHECK(nq_matmul_ex(&pa, U, U, F, 64, &pw, U, U, F, 500, 256, F, 500, DEV, ws_small, nullptr) ==
        NQ_OK);
  CHECK(g_calls.size() == 1 && g_calls[0] == "skinny" && g_last_stages == 3);
  reset();
  CHECK(nq_matmul_ex(&pa, U, U, F, 65, &pw, U, U, F, 500, 256, F, 500, DEV, ws_big, nullptr) ==
        NQ_OK);
  CHECK(g_calls.back() == "decode_once" && g_last_stages == 3);
  reset();
  CHECK(nq_matmul_ex(&pa, U, U, F, 65, &pw, U, U, F, 500, 256, F, 500, DEV, ws_big - 16,
                     nullptr) == NQ_ERR_INVALID_ARG);
  CHECK(g_calls.empty() && mentions("workspace"));
  reset();
  CHECK(nq_matmul_ex(&pa, U, U, F, 65, &pw, U, U, F, 500, 256, F, 500,
                     static_cast<char*>(DEV) + 8, ws_big, nullptr) == NQ_ERR_INVALID_ARG);
  CHECK(g_calls.empty());
  // the int8 contraction needs 2 q m_k <= 127: q = 16, k = 4 does not fit
  nq_params p16 = params(16, 4);
  reset();
  CHECK(nq_matmul_stages(NQ_STAGE_DECODE | NQ_CONTRACT_INT8, &p16, U, U, F, 65, &pw, U, U, F,
                         500, 256, F, 500, DEV, ws_big, nullptr) == NQ_ERR_UNSUPPORTED);
  CHECK(g_calls.empty());
  nq_params p7 = params(7, 4);
  reset();
  CHECK(nq_matmul_stages(NQ_STAGE_DECODE | NQ_CONTRACT_INT8, &p7, U, U, F, 65, &pw, U, U, F,
                         500, 256, F, 500, DEV, ws_big, nullptr) == NQ_OK);
  CHECK(g_last_et == nq::ET_I8 && g_last_stages == (NQ_STAGE_DECODE | NQ_CONTRACT_INT8));
  // rejected shapes
  struct Bad {
    int64_t M, N, K, ldc;
  } bad[] = {{-1, 5, 256, 5}, {3, -1, 256, 5}, {3, 5, 252, 5}, {3, 5, 256, 4},
             {3, 5, 65544, 5}, {(int64_t)1 << 31, 5, 256, 5}};
  for (const Bad& b : bad) {
    reset();
    CHECK(nq_matmul(&pa, U, U, F, b.M, &pw, U, U, F, b.N, b.K, F, b.ldc, nullptr) ==
          NQ_ERR_INVALID_ARG);
    CHECK(g_calls.empty());
  }
  reset();
  CHECK(nq_matmul(&pa, nullptr, U, F, 3, &pw, U, U, F, 5, 256, F, 5, nullptr) ==
        NQ_ERR_INVALID_ARG);
  CHECK(nq_matmul(&pa, U, U, F, 0, &pw, U, U, F, 5, 256, nullptr, 5, nullptr) == NQ_OK);
  CHECK(g_calls.empty());

  // the fused encode-and-multiply: encoder (with W's decode carried for K = 4096), padding,
  // contraction
  const int64_t ws_q = nq_matmul_workspace_size(300, 500, 4096);
  reset();
  CHECK(nq_encode_matmul(0, &pa, DEV, NQ_BF16, 300, 4096, 4096, U, U, F, &pw, U, U, F, 500, F,
                         500, DEV, ws_q, nullptr) == NQ_OK);
  CHECK(g_calls.size() >= 3 && g_calls[0] == "encode_tiles" && g_calls.back() == "decode_once");
  reset();
  CHECK(nq_encode_matmul(NQ_ROTATE_A, &pa, DEV, NQ_BF16, 300, 4096, 4096, U, U, F, &pw, U, U, F,
                         500, F, 500, DEV, ws_q, nullptr) == NQ_OK);
  CHECK(g_calls[0] == "encode_rotated");
  reset();
  CHECK(nq_encode_matmul(NQ_ROTATE_A, &pa, DEV, NQ_BF16, 300, 4000, 4000, U, U, F, &pw, U, U, F,
                         500, F, 500, DEV, ws_q, nullptr) == NQ_ERR_UNSUPPORTED);
  CHECK(g_calls.empty());
}

static void rotate_and_beta() {
  float* Y = F;
  reset();
  CHECK(nq_rotate(DEV, NQ_BF16, 4, 14336, 14336, reinterpret_cast<float*>(0x40000000), 14336,
                  nullptr) == NQ_OK);
  CHECK(g_calls.size() == 2 && g_calls[0] == "rotate_attributes");
  reset();
  CHECK(nq_rotate(DEV, NQ_F32, 4, 4096, 4096, Y, 4096, nullptr) == NQ_ERR_INVALID_ARG);  // overlap
  CHECK(nq_rotate(DEV, NQ_F32, 4, 4000, 4000, Y, 4000, nullptr) == NQ_ERR_UNSUPPORTED);
  CHECK(g_calls.empty());
  reset();
  g_query = hipErrorInvalidDevice;   // the per-device attribute step fails for a new device
  CHECK(nq_rotate(DEV, NQ_BF16, 4, 4096, 4096, reinterpret_cast<float*>(0x40000000), 4096,
                  nullptr) == NQ_ERR_HIP);

  const double betas[3] = {0.1, 0.2, 0.3};
  reset();
  CHECK(nq_beta_stats(16, 0, F, 10, betas, 3, reinterpret_cast<double*>(DEV),
                      static_cast<uint8_t*>(DEV), nullptr) == NQ_OK);
  const double unsorted[3] = {0.2, 0.1, 0.3};
  CHECK(nq_beta_stats(16, 0, F, 10, unsorted, 3, reinterpret_cast<double*>(DEV),
                      static_cast<uint8_t*>(DEV), nullptr) == NQ_ERR_INVALID_ARG);
  const int64_t need = nq_beta_dp_workspace_size(1000, 50);
  CHECK(need == 2 * (50 * 51 / 2 + 50) * 8);
  reset();
  CHECK(nq_beta_dp(reinterpret_cast<double*>(DEV), static_cast<uint8_t*>(DEV), 1000, 50, 4,
                   static_cast<int32_t*>(DEV), reinterpret_cast<double*>(DEV), DEV, need,
                   nullptr) == NQ_OK);
  CHECK(g_calls.size() == 1 && g_calls[0] == "beta_dp");
  reset();
  CHECK(nq_beta_dp(reinterpret_cast<double*>(DEV), static_cast<uint8_t*>(DEV), 1000, 50, 4,
                   static_cast<int32_t*>(DEV), reinterpret_cast<double*>(DEV), DEV, need - 8,
                   nullptr) == NQ_ERR_INVALID_ARG);
  CHECK(g_calls.empty() && mentions("workspace"));
  reset();
  g_launch = hipErrorLaunchFailure;
  CHECK(nq_beta_dp(reinterpret_cast<double*>(DEV), static_cast<uint8_t*>(DEV), 1000, 50, 4,
                   static_cast<int32_t*>(DEV), reinterpret_cast<double*>(DEV), DEV, need,
                   nullptr) == NQ_ERR_HIP);
}

static void per_thread_errors() {
  // nq_last_error belongs to the calling thread
  nq_params p = params();
  nq_params bad = params(99, 4);
  reset();
  CHECK(nq_encode(&bad, DEV, NQ_BF16, 4, 64, 64, U, U, F, nullptr) == NQ_ERR_INVALID_ARG);
  std::string other;
  std::thread t([&] {
    nq_params pb = params(1, 4);
    nq_decode(&pb, U, U, F, 4, 64, DEV, NQ_F16, 64, nullptr);
    other = nq_last_error();
  });
  t.join();
  CHECK(mentions("nq_encode") && other.find("nq_decode") != std::string::npos);
  CHECK(nq_encode(&p, DEV, NQ_BF16, 4, 64, 64, U, U, F, nullptr) == NQ_OK);
  CHECK(std::strcmp(nq_last_error(), "") == 0);
  for (int s = 0; s < 5; ++s) CHECK(nq_status_string((nq_status)s) != nullptr);
  CHECK(nq_codes_words(3, 64) == 24 && nq_beta_words(3, 136) == 6 && nq_codes_words(3, 12) == -1);
}

int main() {
  encode_and_decode();
  matmul_paths();
  rotate_and_beta();
  per_thread_errors();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("all host ABI checks passed\n");
  return 0;
}

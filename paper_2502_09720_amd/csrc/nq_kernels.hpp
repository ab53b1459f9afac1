// Host-side launch interface of the NestQuant kernels (internal to libnestquant.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nestquant.h"

namespace nq {

// The ABI layer's error reporting (nq_last_error) and its product with a workspace, for the
// entry points defined outside nq_api.cpp.
nq_status set_error(nq_status s, const char* fmt, ...);
nq_status matmul_stages(int32_t stages, const nq_params* pa, const uint32_t* a_codes,
                        const uint32_t* a_beta, const float* a_scales, int64_t M,
                        const nq_params* pw, const uint32_t* w_codes, const uint32_t* w_beta,
                        const float* w_scales, int64_t N, int64_t K, float* c, int64_t ldc,
                        void* workspace, int64_t workspace_bytes, void* hip_stream,
                        const char* who);

// The tile decode of one coded operand (tiles_block) carried by wgs extra workgroups of
// another launch; dv is decoder_variant of the operand.  wgs == 0: no task.
struct TileTask {
  const uint32_t* codes;
  const uint32_t* beta;
  int64_t rows;
  int64_t total;   // rows_p * nb_p blocks of the tile
  void* ws;        // the tile
  int nb;
  int nb_p;
  float inv_nbp;   // fl32(1 / nb_p)
  int q;
  uint32_t m2q;
  uint32_t mtab;
  int dv;
  int wgs;
};

struct EncodeArgs {
  int q;           // nesting ratio
  int k;           // number of betas
  float rq;        // fl32(1 / q), estimate for the mod-q reduction
  uint32_t m2q;    // ceil(2^16 / (2q)): floor(X / 2q) = (X * m2q) >> 16 for 0 <= X < 2^11
  uint32_t mq;     // ceil(2^20 / q): floor(u / q) = (u * mq) >> 20 for 0 <= u < 2048 q
  int decoder;     // 0: Alg. 2 / Alg. 5, 1: NestQuantM (App. D)
  int strategy;    // 0: First-beta, 1: Opt-beta (App. F)
  double beta[4];  // fl64(m_t * base), t = 1..4
  // Fused encode-and-multiply: when tiles is set, the decoded tile m_t * X2 of every block
  // is also written to tiles[row * nb_p + j] as the product's decode stage would (ElemType
  // tile_et: 16 B per block for bf16 / fp16, 8 B for int8; mtab as in MatmulOperand).
  void* tiles;
  int tile_et;
  int nb_p;
  uint32_t mtab;
  // With tiles set, the launch of the slot-compacted encoder may also carry W's tile
  // decode, as task.wgs workgroups after the encoder's.
  TileTask task;
  // Rows rotated in LDS before coding (nq_rotate_encode): rot_p = cols / m (m = 1 or 28,
  // 2^rot_lp), rot_s = fl32(1 / sqrt(cols)); rot_p == 0: no rotation.
  int rot_p;
  int rot_lp;
  float rot_s;
};

struct DecodeArgs {
  int q;
  uint32_t m2q;
  int decoder;
  double half_beta[4];  // fl64(t * base) / 2 (exact halving), t = 1..4
};

struct MatmulOperand {
  const uint32_t* codes;
  const uint32_t* beta;
  const float* scales;
  int q;
  uint32_t m2q;
  int64_t rows;
  int decoder;
  uint32_t mtab;   // byte i: the multiple m of base for beta index i (beta = m * base)
};

// Element type of the decoded tiles m * X2 and of the matrix-core instructions: bf16 holds
// every integer up to 256, fp16 up to 2048, int8 up to 127 (all exact).
enum ElemType { ET_BF16 = 0, ET_F16 = 1, ET_I8 = 2 };

hipError_t launch_encode(const void* x, int dtype, int64_t rows, int cols, int64_t ld_x,
                         const EncodeArgs& a, uint32_t* codes, uint32_t* beta, float* scales,
                         hipStream_t st);

hipError_t launch_decode(const uint32_t* codes, const uint32_t* beta, const float* scales,
                         int64_t rows, int cols, void* out, int out_dtype, int64_t ld_out,
                         const DecodeArgs& a, hipStream_t st);

// Stage bits of the launchers: 1 decodes both operands (A's tile and, on the decode-once
// path, W's), 2 contracts; kStageDecodeW decodes only W (A's tile was written by the
// fused encoder).
constexpr int kStageDecodeW = 8;

// The TileTask that decodes operand X into its tile ws (rows_p x nb_p blocks; the element
// type comes with the launch that runs it).
TileTask tile_task(const MatmulOperand& X, int nb, int64_t rows_p, int nb_p, void* ws);
// Whether the encoder of rows of `cols` entries (First-beta) can carry a TileTask, and
// whether it can rotate its rows in LDS (also needs a width nq_rotate supports).
bool encode_carries_task(int cols, int strategy);
bool encode_rotates(int cols, int strategy);
// Where W's tile starts in a decode-once workspace, and its padded shape.
void decode_once_layout(int et, int64_t M, int64_t N, int64_t K, int64_t& w_offset,
                        int64_t& rows_p, int& nb_p);

// Zero the padding of an operand tile written by the fused encoder: rows rows..rows_p-1 and,
// in the first `rows` rows, blocks nb..nb_p-1.
hipError_t launch_tiles_pad(int et, void* ws, int64_t rows, int nb, int64_t rows_p, int nb_p,
                            hipStream_t st);

// Small M (skinny): decode A once into a tile, then decode W straight into MFMA operands.
// stages: bit 0 decodes into the workspace, bit 1 contracts (see nq_matmul_stages); et: the
// ElemType of the tiles and matrix cores (int8: exact int32 sums).
size_t skinny_workspace(int64_t M, int64_t K);
hipError_t launch_matmul_skinny(int stages, int et, const MatmulOperand& A,
                                const MatmulOperand& W, int64_t K, float* c, int64_t ldc,
                                float scale, void* ws, hipStream_t st);

// Decode-once path (large M): workspace bytes, launch (tiles + GEMM), one-time attributes.
size_t decode_once_workspace(int64_t M, int64_t N, int64_t K);
hipError_t launch_matmul_decode_once(int stages, int et, const MatmulOperand& A,
                                     const MatmulOperand& W, int64_t K, float* c, int64_t ldc,
                                     float scale, void* ws, hipStream_t st);
hipError_t gemm_set_attributes();

// No workspace (nq_matmul): each workgroup decodes its own rows' code words into LDS and
// contracts them there (bf16 or fp16 tiles).
hipError_t launch_matmul_fused(int et, const MatmulOperand& A, const MatmulOperand& W,
                               int64_t K, float* c, int64_t ldc, float scale, hipStream_t st);
hipError_t fused_set_attributes();

// Hadamard rotation of rows (nq_rotate): columns 2^k or 28 * 2^k (2^k >= 8), at most this.
constexpr int kRotateMaxCols = 32768;
// m (1 or 28, 0 if unsupported) and p = n / m
int rotation_split(int64_t n, int& p);
hipError_t rotate_set_attributes();
hipError_t launch_rotate(const void* x, int dtype, int64_t rows, int n, int64_t ld_x, float* y,
                         int64_t ld_y, hipStream_t st);

// Beta-set statistics and Alg. 6 (nq_beta): at most 64 candidate betas.
struct BetaGrid {
  int m;
  double beta[64];
};
hipError_t launch_beta_stats(const float* v, int64_t n, const BetaGrid& g, int q, int decoder,
                             double* mse, uint8_t* ov, hipStream_t st);
size_t beta_dp_workspace(int64_t n, int m);
hipError_t launch_beta_dp(const double* mse, const uint8_t* ov, int64_t n, int m, int k,
                          int32_t* chosen, double* loss, void* ws, hipStream_t st);

// M at or below this uses the skinny kernel; above it, decode-once.
constexpr int64_t kFusedMaxM = 64;

// Rows of the product's decoded tiles are padded to whole runs of this many bytes (the
// longest stage row of the decode-once GEMM): 64 bf16 / fp16 values or 128 int8.
constexpr int kTileRowBytes = 128;

// The tile decode (tiles_block) gives each thread this many blocks: one workgroup of 256
// threads per 256 * kTilesPerThread blocks.
constexpr int kTilesPerThread = 4;
inline int64_t tile_workgroups(int64_t total) {
  return (total + 256 * kTilesPerThread - 1) / (256 * kTilesPerThread);
}

// The beta DP's cost sums: a 64-ary tree over the samples; m (m + 1) / 2 transition costs
// and m overload counts per tree node.
constexpr int kBetaFan = 64;
inline int64_t beta_cost_entries(int m) { return (int64_t)m * (m + 1) / 2 + m; }
inline int64_t beta_level2_nodes(int64_t n) {
  return (n + kBetaFan * kBetaFan - 1) / (kBetaFan * kBetaFan);
}

// Launch shape for grid_block: log2 of the lanes per row (-1: 256-block segments) and the
// number of workgroups.
inline void grid_shape(int64_t rows, int nb, int& lg, int64_t& wgs) {
  if (nb <= 256) {
    lg = 0;
    while ((1 << lg) < nb) ++lg;
    const int64_t per = 256 >> lg;
    wgs = (rows + per - 1) / per;
  } else {
    lg = -1;
    wgs = rows * ((nb + 255) / 256);
  }
}

// Decoder kernels by variant: 0 Alg. 2 / Alg. 5, 1 NestQuantM (packed 16-bit), 2 NestQuantM
// at q = 16 (byte SIMD).
__host__ __device__ inline int decoder_variant(int decoder, int q) { return decoder == 0 ? 0 : (q == 16 ? 2 : 1); }

inline uint32_t magic_2q(int q) { return (uint32_t)((65536 + 2 * q - 1) / (2 * q)); }
inline uint32_t magic_q(int q) { return (uint32_t)(((1u << 20) + q - 1) / q); }

}  // namespace nq

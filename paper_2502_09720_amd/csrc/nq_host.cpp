// Host-side helpers of the launchers (no device code): workspace sizes and layouts, the
// descriptor of a carried tile decode, and which row widths the rotation and the fused
// encoder instantiations support.  Kept apart from the kernels so that the C ABI layer and
// these helpers also build with a plain host compiler (the sanitizer build of the ABI tests).
#include <algorithm>

#include "nq_kernels.hpp"

namespace nq {

// Skinny path (M <= 64): only A is decoded into the workspace, rows padded to 16 and to
// kTileRowBytes (64 bf16 / fp16 or 128 int8 values; never more bytes than the 16-bit tile).
size_t skinny_workspace(int64_t M, int64_t K) {
  const int64_t mp = (M + 15) / 16 * 16;
  const int64_t kp = (K + 63) / 64 * 64;
  return (size_t)(mp * kp * 2);
}

// Decode-once path: both tiles, M and N padded to 256 (a multiple of every GEMM tile edge),
// rows to kTileRowBytes.
size_t decode_once_workspace(int64_t M, int64_t N, int64_t K) {
  const int64_t mp = (M + 255) / 256 * 256;
  const int64_t np = (N + 255) / 256 * 256;
  const int64_t kp = (K + 63) / 64 * 64;
  return (size_t)((mp + np) * kp * 2);
}

// Workspace layout of the decode-once path: A's tile (mp x nb_p blocks) then W's (np x nb_p).
void decode_once_layout(int et, int64_t M, int64_t N, int64_t K, int64_t& w_offset,
                        int64_t& rows_p, int& nb_p) {
  const int eb = et == ET_I8 ? 1 : 2;                 // bytes per element
  const int64_t mp = (M + 255) / 256 * 256;
  const int64_t kp = (K * eb + kTileRowBytes - 1) / kTileRowBytes * kTileRowBytes / eb;
  w_offset = mp * kp * eb;
  rows_p = (N + 255) / 256 * 256;
  nb_p = (int)(kp / 8);
}

TileTask tile_task(const MatmulOperand& X, int nb, int64_t rows_p, int nb_p, void* ws) {
  TileTask t;
  t.codes = X.codes;
  t.beta = X.beta;
  t.rows = X.rows;
  t.total = rows_p * nb_p;
  t.ws = ws;
  t.nb = nb;
  t.nb_p = nb_p;
  t.inv_nbp = 1.0f / (float)nb_p;
  t.q = X.q;
  t.m2q = X.m2q;
  t.mtab = X.mtab;
  t.dv = decoder_variant(X.decoder, X.q);
  t.wgs = (int)tile_workgroups(t.total);
  return t;
}

// The beta DP's tree buffers: level 2 (one node per 4096 samples) and level 3, ping-ponged
// upward (every later level fits in one of the two).
size_t beta_dp_workspace(int64_t n, int m) {
  const int64_t Q = beta_cost_entries(m);
  const int64_t a = std::max<int64_t>(beta_level2_nodes(n), 1);
  const int64_t b = (a + kBetaFan - 1) / kBetaFan;
  return (size_t)((a + b) * Q * 8);
}

int rotation_split(int64_t n, int& p) {
  for (int m : {1, 28}) {
    if (n % m) continue;
    const int64_t pp = n / m;
    if (pp >= 8 && (pp & (pp - 1)) == 0 && n <= kRotateMaxCols) {
      p = (int)pp;
      return m;
    }
  }
  return 0;
}

// The encoder instantiations that carry a TileTask: First-beta rows of 257 to 2048 blocks
// (one row per workgroup; every prefill shape of a Llama layer has K in 2056..16384).
bool encode_carries_task(int cols, int strategy) {
  const int nb = cols / 8;
  return strategy == 0 && nb > 256 && nb <= 2048;
}

// The same instantiations rotate their row in LDS, for widths nq_rotate supports:
// 4096, 8192, 16384 and 28 * 2^k = 3584, 7168, 14336.
bool encode_rotates(int cols, int strategy) {
  int p = 0;
  return encode_carries_task(cols, strategy) && rotation_split(cols, p) != 0;
}

}  // namespace nq

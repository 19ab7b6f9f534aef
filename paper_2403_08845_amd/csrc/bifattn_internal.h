// Launch parameters shared by the library's host code and its HIP kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace bifattn {

// Work-group shape of every partial kernel: four 64-wide waves.
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
// Keys per tile: one tile is two 16-key MFMA sub-tiles.
constexpr int kTileKeys = 32;
// Query rows per MFMA N-tile.
constexpr int kRowsPerTile = 16;
// Context path with many query rows per group: work-groups of eight waves,
// one 16-row query tile each.
constexpr int kLargeWaves = 8;
constexpr int kLargeThreads = 64 * kLargeWaves;
constexpr int kLargeRowsPerBlock = kLargeWaves * kRowsPerTile;  // 128
// Largest group size the per-sample decode path holds in registers.
constexpr int kMaxP = 64;
// Lazy softmax rescaling: the running reference maximum is only raised when a
// tile's maximum exceeds it by more than this many powers of two, which keeps
// every weight below 2^kRescaleSlack.
constexpr float kRescaleSlack = 8.0f;
constexpr float kSumBound = 256.0f;  // 2^kRescaleSlack

// Device-side status bits.
constexpr int kStatusLens = 1;
constexpr int kStatusScale = 2;

// Cache element types: bf16, or 8-bit codes (OCP fp8 E4M3, int8) or 4-bit
// codes (int4, two per byte) with per-group scales.
enum KvType { kKvBf16 = 0, kKvFp8 = 1, kKvInt8 = 2, kKvInt4 = 3 };
constexpr int kv_bits(int kv) { return kv == kKvBf16 ? 16 : (kv == kKvInt4 ? 4 : 8); }
// Bytes of one cache row of d elements (d even).
constexpr int kv_row_bytes(int d, int kv) { return d * kv_bits(kv) / 8; }

// Partial result of one query row over one key range, relative to 2^m:
// m  = reference maximum of scale*log2(e)*(q.k) over the range (or -inf),
// l  = sum of 2^(logit - m), acc[d] = sum of 2^(logit - m) * v.
struct PartialsParams {
  const uint16_t* q;
  const uint8_t* Kc;      // caches as bytes: bf16, 8-bit or 4-bit codes
  const uint8_t* Vc;
  const uint8_t* Kd;      // decode cache (replicated cache in ablation mode)
  const uint8_t* Vd;
  const int32_t* lens;
  const float* k_scale;   // [g] key scales, or null for 1
  const float* v_scale;   // [g] value scales, or null (standard path only)
  float* out;             // [b][h][d] rows (standard path only)
  float* ctx_acc;         // [g][S_c][M][d]
  float2* ctx_ml;         // [g][S_c][M]
  float* dec_acc;         // [b][g][S_d][4 waves][p][d]
  float2* dec_ml;         // [b][g][S_d][4 waves][p]
  int* status;
  int b, h, g, p, M;      // h, p count query rows (heads x tokens); M = b*p rows per group
  int ntok;               // new tokens per sample (rows of a unit: head*ntok + token)
  int m_c;
  int m_d_max;            // clamp bound for lens
  int dec_rows;           // row capacity of one (sample, group) decode cache
  int len_offset;         // rows before the decode rows in that cache (0, or m_c in ablation)
  int ctx_keys;           // keys per context work-group (many-row path)
  int S_c;
  int ctx_row_blocks;
  int ctx_wide;           // many-row path: waves of 32 rows per work-group (32x32 MFMA
                          // kernel), or 0 for the kernel of eight 16-row waves
  int dec_keys;           // keys per decode work-group
  int S_d;
  int n_ctx_blocks;       // work-groups of the many-row context path
  int n_ctx_small_blocks; // work-groups of the few-row context path (g * S_c)
  int n_dec_blocks;       // decode work-groups (b * g * S_d); 4 partials each
  float scale_log2;       // |scale| * log2(e); a unit of group gam multiplies in k_scale[gam]
  uint32_t q_sign;        // 0x80008000 when scale < 0 (q enters negated, exactly), else 0
};

struct CombineParams {
  const float* ctx_acc;
  const float2* ctx_ml;
  const float* dec_acc;
  const float2* dec_ml;
  const int32_t* lens;
  const float* k_scale;   // [g] or null: checked here (positive, finite)
  const float* v_scale;   // [g] or null: multiplies the output rows of group g
  float* out;
  int* status;
  int b, h, g, p, M;      // h, p count query rows (heads x tokens)
  int m_d_max;
  int S_c;
  int S_d;
};

// Decode-cache append: the n new rows of every (sample, group).
struct AppendParams {
  const uint8_t* k_new;   // [b][g][n][d] elements of the cache type
  const uint8_t* v_new;
  uint8_t* Kd;            // [b][g][m_d_max][d]
  uint8_t* Vd;
  int32_t* lens;          // [b], advanced by n (capped at m_d_max)
  int* status;
  int b, g, n, m_d_max;
};

enum CtxMode { kCtxNone = 0, kCtxSmall1 = 1, kCtxSmall2 = 2, kCtxSmall4 = 4, kCtxLarge = 8 };

// Events a launch records with its kernel (start / end of the kernel itself,
// not of the stream around it); null members are not recorded.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// XCD-aware order of the many-row context work-groups. Logical id
// chunk * rows + rb is work-group (key chunk, row block rb); the row blocks
// of one chunk read the same keys and should share one XCD's L2. The
// hardware hands dispatch ids to the kXcds XCDs round robin (id % kXcds), so
// XCD x's k-th work-group (id kXcds*k + x) takes row block k % rows of its
// (k / rows)-th chunk among the whole chunks every XCD gets (chunks /
// kXcds of them, consecutive); the ids past those take the remaining chunks
// in order. A bijection of [0, chunks * rows).
constexpr int kXcds = 8;
__host__ __device__ constexpr int xcd_logical(int bid, int chunks, int rows) {
  const int full = chunks / kXcds;  // whole chunks per XCD
  const int x = bid % kXcds, k = bid / kXcds;
  if (k < full * rows) return ((x * full + k / rows) * rows) + k % rows;
  return bid;  // ids from kXcds * full * rows on: the remaining chunks in order
}

// Launch the partial kernel over n_ctx_blocks + n_ctx_small_blocks +
// n_dec_blocks work-groups.
hipError_t launch_partials(const PartialsParams& P, int d, int kv, int ctx_mode, int dec_tiles,
                           hipStream_t stream, const LaunchEvents& ev = {});
hipError_t launch_combine(const CombineParams& C, int d, hipStream_t stream,
                          const LaunchEvents& ev = {});
// Launch the decode-cache append (one work-group per sample).
hipError_t launch_append(const AppendParams& A, int d, int kv, hipStream_t stream,
                         const LaunchEvents& ev = {});
// Launch the standard (unsplit) attention kernel: one work-group per
// (sample, group), `tiles` 16-row query tiles per wave, output written directly.
hipError_t launch_standard(const PartialsParams& P, int d, int kv, int tiles, hipStream_t stream,
                           const LaunchEvents& ev = {});
// Fixed device scratch of the allocation-free entry point: one copy per
// device, held from the library's load to the end of the process.
constexpr size_t kScratchBytes = size_t(64) << 20;
// Device address of `device`'s scratch copy (looked up once per device, with
// that device current; later calls return the cached address).
hipError_t scratch_address(int device, void** ptr);

// Launch the many-row context kernel over n_ctx_blocks work-groups.
hipError_t launch_ctx_large(const PartialsParams& P, int d, int kv, hipStream_t stream,
                            const LaunchEvents& ev = {});

}  // namespace bifattn

// HIP kernels of libbifattn for gfx950 (CDNA4, wave64, bf16 MFMA 16x16x32).
//
// Bifurcated attention (Section 4.2): the logits of one query token split
// along the key axis into a context part <q, K_c> and a decode part
// <q, K_d> (Eq. 3); the weighted values split the same way and are summed
// (Eq. 4); one softmax spans both. Here each work-group turns one key range
// into an online-softmax partial (m, l, acc) for each of its query rows, and
// the combine kernel merges all partials of a row into the exact softmax
// result. The context part reads each K_c/V_c tile once per group and applies
// it to all b*p query rows of that group; that single read is the IO saving
// of Section 4.3.
//
// MFMA operand layouts used throughout (v_mfma_f32_16x16x32_bf16, lane l,
// n = l & 15, G = l >> 4):
//   A (16 x 32): lane holds A[n][8G .. 8G+7]
//   B (32 x 16): lane holds B[8G .. 8G+7][n]
//   C (16 x 16): lane holds C[4G .. 4G+3][n]
// Logits are computed transposed, S^T = K Q^T, so that a lane's 8 logits are
// one query row n and keys 8G..8G+7 -- exactly the B operand of the value
// product O^T = V^T P^T. Within a 32-key tile, QK sub-tile a (0/1) puts key
// 8*(r>>2) + 4a + (r&3) on MFMA row r; the accumulator of sub-tile a then
// holds keys 8G+4a .. 8G+4a+3. V^T operands are built from value rows by a
// per-lane 16-bit transpose; dimension block t of the output holds dims
// DV*r + t (DV = d/16), so lane (n, G) ends up owning output dims
// [4*DV*G, 4*DV*G + 4*DV) of query row n.
#include <hip/hip_runtime.h>

#include "bifattn_internal.h"

namespace bifattn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x4 mfma_bf16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v = {(__bf16)lo, (__bf16)hi};  // round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Value row slice a lane loads: DV consecutive bf16 (16 B for d=128, 8 B for d=64).
template <int D> struct VSlice;
template <> struct VSlice<128> {
  typedef u32x4 type;
  static __device__ __forceinline__ type load(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
  }
  static __device__ __forceinline__ type zero() { return u32x4{0, 0, 0, 0}; }
};
template <> struct VSlice<64> {
  typedef u32x2 type;
  static __device__ __forceinline__ type load(const uint16_t* p) {
    return *reinterpret_cast<const u32x2*>(p);
  }
  static __device__ __forceinline__ type zero() { return u32x2{0, 0}; }
};

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Row r of a QK sub-tile a holds tile key 8*(r>>2) + 4a + (r&3).
__device__ __forceinline__ int qk_key(int a, int r) { return 8 * (r >> 2) + 4 * a + (r & 3); }

// Element t of a value slice: 16-bit lane t of the slice's words.
template <typename S>
__device__ __forceinline__ uint32_t vword(const S& s, int t) { return s[t >> 1]; }

// Pack element t of two value rows (even key, odd key) into one 32-bit word.
__device__ __forceinline__ uint32_t pair_elem(uint32_t even_w, uint32_t odd_w, int t) {
  return (t & 1) ? ((even_w >> 16) | (odd_w & 0xffff0000u))
                 : ((even_w & 0xffffu) | (odd_w << 16));
}

// Per-wave running state of NT query tiles.
template <int D, int NT> struct RowState {
  static constexpr int DV = D / 16;
  float mref[NT];       // reference maximum (log2 units), uniform over the row's 4 lanes
  float l[NT];          // this lane's share of the row sum
  f32x4 acc[NT][DV];    // O^T accumulators
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      mref[nt] = kNegInf;
      l[nt] = 0.f;
#pragma unroll
      for (int t = 0; t < DV; ++t) acc[nt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

// One 32-key tile against NT query tiles: S^T = K Q^T on MFMA, online softmax
// with lazy rescaling, O^T += V^T P^T on MFMA. kop/vop are this lane's K and
// V^T operands, qop[nt][s] the Q^T operands. Keys >= nvalid are masked.
template <int D, int NT>
__device__ __forceinline__ void tile_update(RowState<D, NT>& st, const u32x4 (&kop)[2][D / 32],
                                            const u32x4 (&vop)[D / 16],
                                            const u32x4 (&qop)[NT][D / 32], int nvalid,
                                            float scale_log2, int lane) {
  constexpr int KS = D / 32;
  constexpr int DV = D / 16;
  const int G = lane >> 4;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      s0 = mfma_bf16(kop[0][s], qop[nt][s], s0);
      s1 = mfma_bf16(kop[1][s], qop[nt][s], s1);
    }
    float x[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = s0[j] * scale_log2;
      x[4 + j] = s1[j] * scale_log2;
    }
    if (nvalid < kTileKeys) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * G + e >= nvalid) x[e] = kNegInf;
    }
    float tmax = x[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) tmax = fmaxf(tmax, x[e]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const bool raise = tmax > st.mref[nt] + kRescaleSlack;
    if (__any(raise)) {
      // Rows that do not raise keep alpha = 1 (and never form -inf - -inf).
      const float alpha = raise ? exp2_fast(st.mref[nt] - tmax) : 1.f;  // 0 when mref = -inf
      st.l[nt] *= alpha;
#pragma unroll
      for (int t = 0; t < DV; ++t) st.acc[nt][t] *= alpha;
      st.mref[nt] = raise ? tmax : st.mref[nt];
    }
    const float base = st.mref[nt] == kNegInf ? 0.f : st.mref[nt];
    float pr[8];
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pr[e] = exp2_fast(x[e] - base);
      psum += pr[e];
    }
    st.l[nt] += psum;
    u32x4 pb;
#pragma unroll
    for (int w = 0; w < 4; ++w) pb[w] = pack_bf16(pr[2 * w], pr[2 * w + 1]);
#pragma unroll
    for (int t = 0; t < DV; ++t) st.acc[nt][t] = mfma_bf16(vop[t], pb, st.acc[nt][t]);
  }
}

// Q^T operands of NT query tiles. row_ptr(r) gives the bf16 row of tile row r
// (r = nt*16 + n) or nullptr when the row is padding.
template <int D, int NT, typename RowPtr>
__device__ __forceinline__ void load_q(u32x4 (&qop)[NT][D / 32], RowPtr row_ptr, int lane) {
  const int n = lane & 15, G = lane >> 4;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const uint16_t* qr = row_ptr(nt * kRowsPerTile + n);
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      qop[nt][s] = qr ? load16(qr + s * 32 + G * 8) : u32x4{0, 0, 0, 0};
  }
}

// Register path: one wave loads a whole 32-key tile into its own operands.
template <int D>
__device__ __forceinline__ void load_tile_regs(u32x4 (&kop)[2][D / 32], u32x4 (&vop)[D / 16],
                                               const uint16_t* K, const uint16_t* V, int nvalid,
                                               int lane) {
  constexpr int KS = D / 32;
  constexpr int DV = D / 16;
  typedef typename VSlice<D>::type VS;
  const int r = lane & 15, G = lane >> 4;
  VS vrow[8];
  if (nvalid >= kTileKeys) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const uint16_t* kp = K + (size_t)qk_key(a, r) * D + G * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) kop[a][s] = load16(kp + s * 32);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) vrow[e] = VSlice<D>::load(V + (size_t)(8 * G + e) * D + DV * r);
  } else {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int key = qk_key(a, r);
      const uint16_t* kp = K + (size_t)key * D + G * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) kop[a][s] = key < nvalid ? load16(kp + s * 32) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = 8 * G + e;
      vrow[e] = key < nvalid ? VSlice<D>::load(V + (size_t)key * D + DV * r) : VSlice<D>::zero();
    }
  }
#pragma unroll
  for (int t = 0; t < DV; ++t)
#pragma unroll
    for (int w = 0; w < 4; ++w)
      vop[t][w] = pair_elem(vword(vrow[2 * w], t), vword(vrow[2 * w + 1], t), t);
}

// Row totals of the per-lane sums (the four lanes of a row share the row).
template <int D, int NT>
__device__ __forceinline__ void finish_sums(RowState<D, NT>& st) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    st.l[nt] += __shfl_xor(st.l[nt], 16);
    st.l[nt] += __shfl_xor(st.l[nt], 32);
  }
}

// Merge the four waves' states of the same NT*16 rows through LDS (in wave
// order, so the result is deterministic) and write rows < nrows to
// acc_out[row * row_stride_acc] / ml_out[row * row_stride_ml].
template <int D, int NT>
__device__ __forceinline__ void merge_waves_and_store(RowState<D, NT>& st, float* lds, int nrows,
                                                      float* acc_out, size_t row_stride_acc,
                                                      float2* ml_out, size_t row_stride_ml) {
  constexpr int DV = D / 16;
  constexpr int LD = D + 4;  // padded LDS row
  constexpr int ROWS = NT * kRowsPerTile;
  float* acc_s = lds;
  float* m_s = lds + ROWS * LD;
  float* l_s = m_s + ROWS;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, G = lane >> 4;
  finish_sums(st);
  for (int turn = 0; turn < kWaves; ++turn) {
    if (wave == turn) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int row = nt * kRowsPerTile + n;
        const float mo = turn ? m_s[row] : kNegInf;
        const float lo = turn ? l_s[row] : 0.f;
        const float mn = fmaxf(mo, st.mref[nt]);
        const float base = mn == kNegInf ? 0.f : mn;
        const float fa = exp2_fast(mo - base), fb = exp2_fast(st.mref[nt] - base);
        float* arow = acc_s + row * LD;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float* dst = arow + DV * (4 * G + j);
#pragma unroll
          for (int t4 = 0; t4 < DV; t4 += 4) {
            f32x4 old = turn ? *reinterpret_cast<f32x4*>(dst + t4) : f32x4{0.f, 0.f, 0.f, 0.f};
            f32x4 mine = {st.acc[nt][t4][j], st.acc[nt][t4 + 1][j], st.acc[nt][t4 + 2][j],
                          st.acc[nt][t4 + 3][j]};
            *reinterpret_cast<f32x4*>(dst + t4) = old * fa + mine * fb;
          }
        }
        if (G == 0) {
          m_s[row] = mn;
          l_s[row] = lo * fa + st.l[nt] * fb;
        }
      }
    }
    __syncthreads();
  }
  // Cooperative copy of the valid rows to the workspace.
  constexpr int V4 = D / 4;
  for (int idx = threadIdx.x; idx < nrows * V4; idx += kThreads) {
    const int row = idx / V4, c = idx % V4;
    *reinterpret_cast<f32x4*>(acc_out + row * row_stride_acc + 4 * c) =
        *reinterpret_cast<const f32x4*>(acc_s + row * LD + 4 * c);
  }
  for (int row = threadIdx.x; row < nrows; row += kThreads)
    ml_out[row * row_stride_ml] = float2{m_s[row], l_s[row]};
}

__device__ __forceinline__ int clamp_len(const int32_t* lens, int i, int m_d_max) {
  const int raw = lens ? lens[i] : 0;
  return raw < 0 ? 0 : (raw > m_d_max ? m_d_max : raw);
}

// ---------------------------------------------------------------------------
// Decode part (and the replicated ablation): work-group (sample i, group gam,
// key split s) over the sample's own cache rows [s*dec_keys, ...). Query rows
// are the p heads of group gam. Waves take interleaved tiles and merge.
template <int D, int NT>
__device__ void decode_block(const PartialsParams& P, int blk, float* lds) {
  const int s = blk % P.S_d;
  const int ig = blk / P.S_d;
  const int gam = ig % P.g, i = ig / P.g;
  const int total = P.len_offset + clamp_len(P.lens, i, P.m_d_max);
  const int k0 = s * P.dec_keys;
  if (k0 >= total) return;  // whole work-group: nothing to do for this split
  const int k1 = min(total, k0 + P.dec_keys);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t cache = (size_t)(i * P.g + gam) * P.dec_rows * D;
  const uint16_t* Kb = P.Kd + cache;
  const uint16_t* Vb = P.Vd + cache;
  u32x4 qop[NT][D / 32];
  const uint16_t* qbase = P.q + ((size_t)i * P.h + (size_t)gam * P.p) * D;
  const int p = P.p;
  load_q<D, NT>(qop, [&](int r) -> const uint16_t* { return r < p ? qbase + (size_t)r * D : nullptr; },
                lane);
  RowState<D, NT> st;
  st.init();
  for (int key0 = k0 + wave * kTileKeys; key0 < k1; key0 += kWaves * kTileKeys) {
    u32x4 kop[2][D / 32];
    u32x4 vop[D / 16];
    const int nvalid = min(kTileKeys, k1 - key0);
    load_tile_regs<D>(kop, vop, Kb + (size_t)key0 * D, Vb + (size_t)key0 * D, nvalid, lane);
    tile_update<D, NT>(st, kop, vop, qop, nvalid, P.scale_log2, lane);
  }
  const size_t prow = ((size_t)ig * P.S_d + s) * P.p;
  merge_waves_and_store<D, NT>(st, lds, p, P.dec_acc + prow * D, D, P.dec_ml + prow, 1);
}

// Context part, few query rows per group (M = b*p <= 64): work-group
// (group gam, key split s) reads Kc/Vc rows [s*ctx_keys, ...) once, each tile
// straight into the operands of the wave that uses it for all M rows.
template <int D, int NT>
__device__ void ctx_small_block(const PartialsParams& P, int blk, float* lds) {
  const int s = blk % P.S_c, gam = blk / P.S_c;
  const int k0 = s * P.ctx_keys;
  const int k1 = min(P.m_c, k0 + P.ctx_keys);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t cache = (size_t)gam * P.m_c * D;
  const uint16_t* Kb = P.Kc + cache;
  const uint16_t* Vb = P.Vc + cache;
  const int M = P.M, p = P.p, h = P.h;
  const uint16_t* q = P.q;
  u32x4 qop[NT][D / 32];
  load_q<D, NT>(qop, [&](int r) -> const uint16_t* {
    if (r >= M) return nullptr;
    const int i = r / p, jp = r - i * p;
    return q + ((size_t)i * h + (size_t)gam * p + jp) * D;
  }, lane);
  RowState<D, NT> st;
  st.init();
  for (int key0 = k0 + wave * kTileKeys; key0 < k1; key0 += kWaves * kTileKeys) {
    u32x4 kop[2][D / 32];
    u32x4 vop[D / 16];
    const int nvalid = min(kTileKeys, k1 - key0);
    load_tile_regs<D>(kop, vop, Kb + (size_t)key0 * D, Vb + (size_t)key0 * D, nvalid, lane);
    tile_update<D, NT>(st, kop, vop, qop, nvalid, P.scale_log2, lane);
  }
  const size_t prow = ((size_t)gam * P.S_c + s) * P.M;
  merge_waves_and_store<D, NT>(st, lds, M, P.ctx_acc + prow * D, D, P.ctx_ml + prow, 1);
}

// Context part, many query rows per group: work-group (group gam, key split
// s, row block rb) of 256 query rows. Each 32-key tile of Kc/Vc is loaded
// from HBM once per work-group into LDS, already in MFMA operand order (the
// V^T transpose is done once, on the way in), and all four waves read it for
// their 64 rows. Double-buffered: the next tile's global loads are in flight
// while the current one is consumed. Row blocks of one key chunk are
// scheduled on the same XCD so that they share its L2.
template <int D>
__device__ void ctx_large_block(const PartialsParams& P, int blk, float* lds) {
  constexpr int KS = D / 32;
  constexpr int DV = D / 16;
  constexpr int NT = kLargeTilesPerWave;
  constexpr int KOPS = 2 * KS;             // K operands per tile
  constexpr int KPW = KOPS / kWaves;       // K operands each wave stages
  constexpr int OPS = KOPS + DV;           // operands per tile (16 B per lane each)
  typedef typename VSlice<D>::type VS;
  const int rb = blk % P.ctx_row_blocks;
  const int sg = blk / P.ctx_row_blocks;
  const int s = sg % P.S_c, gam = sg / P.S_c;
  const int k0 = s * P.ctx_keys;
  const int k1 = min(P.m_c, k0 + P.ctx_keys);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, G = lane >> 4;
  const size_t cache = (size_t)gam * P.m_c * D;
  const uint16_t* Kb = P.Kc + cache;
  const uint16_t* Vb = P.Vc + cache;
  const int M = P.M, p = P.p, h = P.h;
  const int row0 = rb * kLargeRowsPerBlock + wave * NT * kRowsPerTile;
  const uint16_t* q = P.q;
  u32x4 qop[NT][KS];
  load_q<D, NT>(qop, [&](int rr) -> const uint16_t* {
    const int row = row0 + rr;
    if (row >= M) return nullptr;
    const int i = row / p, jp = row - i * p;
    return q + ((size_t)i * h + (size_t)gam * p + jp) * D;
  }, lane);
  // LDS: two buffers of OPS operand slots x 64 lanes x 16 B.
  u32x4* opbuf = reinterpret_cast<u32x4*>(lds);
  auto slot = [&](int buf, int op) -> u32x4* { return opbuf + ((size_t)buf * OPS + op) * 64; };

  // Staging registers of the next tile: this wave's K operands and two value rows.
  u32x4 kst[KPW];
  VS vst[2];
  auto fetch = [&](int key0) {
    const int nvalid = min(kTileKeys, k1 - key0);
#pragma unroll
    for (int c = 0; c < KPW; ++c) {
      const int op = wave * KPW + c, a = op / KS, ss = op % KS;
      const int key = qk_key(a, r);
      kst[c] = key < nvalid ? load16(Kb + (size_t)(key0 + key) * D + ss * 32 + G * 8)
                            : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int key = 8 * G + 2 * wave + c;
      vst[c] = key < nvalid ? VSlice<D>::load(Vb + (size_t)(key0 + key) * D + DV * r)
                            : VSlice<D>::zero();
    }
  };
  auto stage = [&](int buf) {
#pragma unroll
    for (int c = 0; c < KPW; ++c) slot(buf, wave * KPW + c)[lane] = kst[c];
    // word `wave` of V^T operand t = keys (8G + 2*wave, 8G + 2*wave + 1) at dim DV*r + t
#pragma unroll
    for (int t = 0; t < DV; ++t)
      reinterpret_cast<uint32_t*>(slot(buf, KOPS + t) + lane)[wave] =
          pair_elem(vword(vst[0], t), vword(vst[1], t), t);
  };

  RowState<D, NT> st;
  st.init();
  const int ntiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  fetch(k0);
  stage(0);
  __syncthreads();
  for (int it = 0; it < ntiles; ++it) {
    const int buf = it & 1;
    if (it + 1 < ntiles) fetch(k0 + (it + 1) * kTileKeys);
    u32x4 kop[2][KS];
    u32x4 vop[DV];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int ss = 0; ss < KS; ++ss) kop[a][ss] = slot(buf, a * KS + ss)[lane];
#pragma unroll
    for (int t = 0; t < DV; ++t) vop[t] = slot(buf, KOPS + t)[lane];
    const int nvalid = min(kTileKeys, k1 - (k0 + it * kTileKeys));
    tile_update<D, NT>(st, kop, vop, qop, nvalid, P.scale_log2, lane);
    if (it + 1 < ntiles) stage(buf ^ 1);
    __syncthreads();
  }
  finish_sums(st);
  const size_t pbase = ((size_t)gam * P.S_c + s) * P.M;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int row = row0 + nt * kRowsPerTile + r;
    if (row < M) {
      float* dst = P.ctx_acc + (pbase + row) * D + 4 * DV * G;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int t4 = 0; t4 < DV; t4 += 4)
          *reinterpret_cast<f32x4*>(dst + DV * j + t4) =
              f32x4{st.acc[nt][t4][j], st.acc[nt][t4 + 1][j], st.acc[nt][t4 + 2][j],
                    st.acc[nt][t4 + 3][j]};
      if (G == 0) P.ctx_ml[pbase + row] = float2{st.mref[nt], st.l[nt]};
    }
  }
}

template <int D, int NT> struct MergeLds {
  static constexpr int bytes = (NT * kRowsPerTile * (D + 4) + 2 * NT * kRowsPerTile) * 4;
};
template <int D> struct LargeLds {
  static constexpr int bytes = 2 * (2 * (D / 32) + D / 16) * 64 * 16;
};
constexpr int cmax(int a, int b) { return a > b ? a : b; }

// XCD-aware order for the large context path: the hardware hands work-group
// ids to the 8 XCDs round robin, so logical ids that must share an L2 (the
// row blocks of one key chunk) are spread with stride 8 in dispatch order.
__device__ __forceinline__ int xcd_logical(int bid, int n) {
  constexpr int X = 8;
  const int per = n / X;
  if (bid >= per * X) return bid;  // ragged remainder keeps its id
  return (bid % X) * per + bid / X;
}

template <int D, int CTX, int NTD>
__global__ __launch_bounds__(kThreads) void partials_kernel(PartialsParams P) {
  constexpr int LDS_CTX = CTX == kCtxLarge ? LargeLds<D>::bytes
                          : CTX == kCtxNone ? 0 : MergeLds<D, (CTX > 0 ? CTX : 1)>::bytes;
  constexpr int LDS = cmax(cmax(LDS_CTX, MergeLds<D, NTD>::bytes), 16);
  __shared__ __attribute__((aligned(16))) float lds[LDS / 4];
  const int bid = blockIdx.x;
  if (bid < P.n_ctx_blocks) {
    if constexpr (CTX == kCtxLarge) {
      ctx_large_block<D>(P, xcd_logical(bid, P.n_ctx_blocks), lds);
    } else if constexpr (CTX != kCtxNone) {
      ctx_small_block<D, CTX>(P, bid, lds);
    }
  } else {
    decode_block<D, NTD>(P, bid - P.n_ctx_blocks, lds);
  }
}

// Combine (the joint softmax of Eq. 3-4): one wave per output row (i, j)
// merges the row's context partials (group j/p, every split) and decode
// partials (sample i, group j/p, the splits that hold keys) into
// out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k, M = max_k m_k.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(CombineParams C) {
  constexpr int PER = D / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = blockIdx.x * 4 + wave;
  if (row >= C.b * C.h) return;
  const int i = row / C.h, j = row - i * C.h;
  const int gam = j / C.p, jp = j - gam * C.p;
  const int raw = C.lens ? C.lens[i] : 0;
  const int len = clamp_len(C.lens, i, C.m_d_max);
  if (raw != len && j == 0 && lane == 0) atomicOr(C.status, kStatusLens);
  const int total = C.len_offset + len;
  const int nsd = C.S_d ? (total + C.dec_keys - 1) / C.dec_keys : 0;
  const int np = C.S_c + nsd;
  const size_t cbase = (size_t)gam * C.S_c * C.M + (size_t)i * C.p + jp;  // + k*M
  const size_t dbase = ((size_t)(i * C.g + gam) * C.S_d) * C.p + jp;      // + k*p
  auto idx = [&](int k) -> size_t {
    return k < C.S_c ? cbase + (size_t)k * C.M : dbase + (size_t)(k - C.S_c) * C.p;
  };
  auto ml = [&](int k) -> float2 { return k < C.S_c ? C.ctx_ml[idx(k)] : C.dec_ml[idx(k)]; };
  auto accp = [&](int k) -> const float* {
    return (k < C.S_c ? C.ctx_acc : C.dec_acc) + idx(k) * D;
  };
  float mx = kNegInf;
  for (int k = lane; k < np; k += 64) mx = fmaxf(mx, ml(k).x);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  const float base = mx == kNegInf ? 0.f : mx;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  float L = 0.f;
  for (int k = 0; k < np; ++k) {
    const float2 v = ml(k);
    const float w = exp2_fast(v.x - base);
    L += w * v.y;
    const float* a = accp(k) + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += w * a[e];
  }
  float* o = C.out + (size_t)row * D + lane * PER;
  const float inv = 1.f / L;
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = acc[e] * inv;
}

template <int D, int CTX>
hipError_t launch_partials_ctx(const PartialsParams& P, int dec_tiles, hipStream_t stream) {
  const int grid = P.n_ctx_blocks + P.n_dec_blocks;
  if (grid == 0) return hipSuccess;
  switch (dec_tiles) {
    case 1: partials_kernel<D, CTX, 1><<<grid, kThreads, 0, stream>>>(P); break;
    case 2: partials_kernel<D, CTX, 2><<<grid, kThreads, 0, stream>>>(P); break;
    case 4: partials_kernel<D, CTX, 4><<<grid, kThreads, 0, stream>>>(P); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_partials_d(const PartialsParams& P, int ctx_mode, int dec_tiles,
                             hipStream_t stream) {
  switch (ctx_mode) {
    case kCtxNone: return launch_partials_ctx<D, kCtxNone>(P, dec_tiles, stream);
    case kCtxSmall1: return launch_partials_ctx<D, kCtxSmall1>(P, dec_tiles, stream);
    case kCtxSmall2: return launch_partials_ctx<D, kCtxSmall2>(P, dec_tiles, stream);
    case kCtxSmall4: return launch_partials_ctx<D, kCtxSmall4>(P, dec_tiles, stream);
    case kCtxLarge: return launch_partials_ctx<D, kCtxLarge>(P, dec_tiles, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_partials(const PartialsParams& P, int d, int ctx_mode, int dec_tiles,
                           hipStream_t stream) {
  if (d == 128) return launch_partials_d<128>(P, ctx_mode, dec_tiles, stream);
  if (d == 64) return launch_partials_d<64>(P, ctx_mode, dec_tiles, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const CombineParams& C, int d, hipStream_t stream) {
  const int rows = C.b * C.h;
  const int grid = (rows + 3) / 4;
  if (d == 128)
    combine_kernel<128><<<grid, 256, 0, stream>>>(C);
  else if (d == 64)
    combine_kernel<64><<<grid, 256, 0, stream>>>(C);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace bifattn

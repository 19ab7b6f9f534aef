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
// Logits are computed transposed, S^T = K Q^T: query rows are the MFMA
// columns, so all logits a lane holds belong to one query row n. Within a
// 32-key tile, row r of QK sub-tile a (0/1) is tile key 16a + 4(r&3) + (r>>2)
// (qk_key); the accumulators of the two sub-tiles then give lane (n, G) the
// logits of keys 4e + G, e = 0..7. After the softmax those 8 weights, packed
// to bf16, are the lane's B operand of the value product O^T = V^T P^T, whose
// k-slot (G, e) is key 4e + G; the lane builds its V^T operand from the same
// value rows 4e + G (a 16-bit transpose inside the lane), so both operands
// agree on the key of every k-slot. Dimension block t of the output holds
// dims DV*m + t on MFMA row m (DV = d/16), so lane (n, G) ends up owning
// output dims [4*DV*G, 4*DV*G + 4*DV) of query row n.
//
// Caches may hold 8-bit codes (OCP fp8 E4M3 or int8) or 4-bit codes (int4,
// two per byte), with one scale per KV group for keys and one for values:
// every code value is exactly a bf16 value, so codes are widened to bf16 on
// the way from memory to the operands and the matrix products stay bf16. The key scale folds into the softmax scale of
// the group's units and the value scale into the combine.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <mutex>

#include "bifattn_internal.h"

namespace bifattn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;  // LDS-qualified operand slot

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

// Cross-row exchanges without a trip through LDS: v_permlane16_swap and
// v_permlane32_swap of a register with itself return, in their two results,
// the lane's own value and the value of lane l^16 (l^32), in an order that
// depends on the row; max / sum of the two is the same in every lane. The
// two vector elements are copied to scalars before the float reinterpret:
// __builtin_bit_cast applied to an element of the result vector reads
// element 0 whatever the index.
template <bool kWide>
__device__ __forceinline__ void swap_halves(float x, float& a, float& b) {
  const unsigned u = __float_as_uint(x);
  const auto r = kWide ? __builtin_amdgcn_permlane32_swap(u, u, false, false)
                       : __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const unsigned r0 = r[0], r1 = r[1];
  a = __uint_as_float(r0);
  b = __uint_as_float(r1);
}
__device__ __forceinline__ float xor16_max(float x) {
  float a, b;
  swap_halves<false>(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float xor32_max(float x) {
  float a, b;
  swap_halves<true>(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float xor16_sum(float x) {
  float a, b;
  swap_halves<false>(x, a, b);
  return a + b;
}
__device__ __forceinline__ float xor32_sum(float x) {
  float a, b;
  swap_halves<true>(x, a, b);
  return a + b;
}
// Whole-wave reductions: permlane swaps across rows, then shuffles in a row.
__device__ __forceinline__ float wave_max(float x) {
  x = xor32_max(xor16_max(x));
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
  x = xor32_sum(xor16_sum(x));
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// Wave index within the work-group, as a wave-uniform (scalar) value so that
// branches on it and on tile bounds derived from it stay scalar.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// Byte offsets into a buffer resource are formed in 32-bit unsigned
// arithmetic: prefetches past the end of a cache near the 2^31-byte limit may
// wrap, which is well defined here and lands outside the resource's range
// (or inside it, on bytes that are never consumed), where a raw buffer load
// returns zeros or valid memory and never faults.
__device__ __forceinline__ int boff(uint32_t x) { return __builtin_bit_cast(int, x); }

// Cache policy of the loads that stream a cache: every byte of the decode
// cache, and of the context on the few-row path, is read exactly once per
// step, so those loads are non-temporal (the nt bit: streamed past the caches
// instead of displacing lines). Measured on MI355X over 402 MB of loads-only
// regions: 6.0 TB/s with the default policy, 6.7 TB/s with nt.
constexpr int kAuxStream = 2;

// N bytes a lane loads with one buffer instruction (cache policy AUX), and
// 32-bit word w of them.
template <int N> struct Raw;
template <> struct Raw<16> {
  typedef u32x4 type;
  template <int AUX = 0>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX);
  }
  static __device__ __forceinline__ type zero() { return u32x4{0, 0, 0, 0}; }
  static __device__ __forceinline__ uint32_t word(const type& v, int w) { return v[w]; }
};
template <> struct Raw<8> {
  typedef u32x2 type;
  template <int AUX = 0>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX);
  }
  static __device__ __forceinline__ type zero() { return u32x2{0, 0}; }
  static __device__ __forceinline__ uint32_t word(const type& v, int w) { return v[w]; }
};
template <> struct Raw<4> {
  typedef uint32_t type;
  template <int AUX = 0>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX);
  }
  static __device__ __forceinline__ type zero() { return 0u; }
  static __device__ __forceinline__ uint32_t word(const type& v, int) { return v; }
};
template <> struct Raw<2> {
  typedef uint32_t type;
  template <int AUX = 0>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, AUX);
  }
  static __device__ __forceinline__ type zero() { return 0u; }
  static __device__ __forceinline__ uint32_t word(const type& v, int) { return v; }
};
template <> struct Raw<1> {
  typedef uint32_t type;
  template <int AUX = 0>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b8(r, off, 0, AUX);
  }
  static __device__ __forceinline__ type zero() { return 0u; }
  static __device__ __forceinline__ uint32_t word(const type& v, int) { return v; }
};

// Pack element t of two bf16 value rows (even key, odd key) into one word.
__device__ __forceinline__ uint32_t pair_elem(uint32_t even_w, uint32_t odd_w, int t) {
  return (t & 1) ? ((even_w >> 16) | (odd_w & 0xffff0000u))
                 : ((even_w & 0xffffu) | (odd_w << 16));
}

// Cache element codecs. BITS: bits per element; bytes(n): bytes of n
// elements. For the 8-bit codes, lo(w) / hi(w) widen codes 0-1 / 2-3 of a
// word to a bf16 pair (code 0 or 2 in the low half); for every code type
// pair(e, o, t) widens code t of word e and code t of word o. The
// conversions are exact: an fp8 E4M3 value has 4 significant bits, an int8
// value 8 and an int4 value 4, all inside bf16's exponent range.
template <int B> struct KvBits {
  static constexpr int BITS = B;
  static constexpr int bytes(int n) { return n * B / 8; }
};
struct KvBf16 : KvBits<16> {
  static __device__ __forceinline__ uint32_t pair(uint32_t e, uint32_t o, int t) {
    return pair_elem(e, o, t);
  }
};
struct KvFp8 : KvBits<8> {
  static __device__ __forceinline__ uint32_t lo(uint32_t w) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, false));
  }
  static __device__ __forceinline__ uint32_t hi(uint32_t w) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, true));
  }
  static __device__ __forceinline__ uint32_t pair(uint32_t e, uint32_t o, int t) {
    // v_perm_b32: selectors 0-3 take bytes of the second operand (e), 4-7 of
    // the first (o), 12 gives zero.
    return lo(__builtin_amdgcn_perm(o, e, 0x0C0C0000u | ((4u + t) << 8) | (uint32_t)t));
  }
};
struct KvInt8 : KvBits<8> {
  static __device__ __forceinline__ float code(uint32_t w, int t) {
    return (float)(signed char)(w >> (8 * t));
  }
  // Two integral floats of at most 8 significant bits: their upper halves
  // are their bf16 values.
  static __device__ __forceinline__ uint32_t two(float a, float b) {
    return __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
  }
  static __device__ __forceinline__ uint32_t lo(uint32_t w) { return two(code(w, 0), code(w, 1)); }
  static __device__ __forceinline__ uint32_t hi(uint32_t w) { return two(code(w, 2), code(w, 3)); }
  static __device__ __forceinline__ uint32_t pair(uint32_t e, uint32_t o, int t) {
    return two(code(e, t), code(o, t));
  }
};
// Two's complement 4-bit codes, eight to a word: element 2u of a row in the
// low nibble of its byte u, so nibble t of a word is element t of the word's
// eight.
struct KvInt4 : KvBits<4> {
  static __device__ __forceinline__ float code(uint32_t w, int t) {
    return (float)((int)(w << (28 - 4 * t)) >> 28);  // sign-extended nibble t
  }
  static __device__ __forceinline__ uint32_t pair(uint32_t e, uint32_t o, int t) {
    return KvInt8::two(code(e, t), code(o, t));
  }
};

// 8 cache elements -> 8 bf16 (one MFMA operand): 16 raw bytes (bf16) as
// they are, or 8 codes widened.
template <typename KV> struct Widen8;
template <> struct Widen8<KvBf16> {
  static __device__ __forceinline__ u32x4 run(const u32x4& r) { return r; }
};
template <typename C> struct Widen8Codes {
  static __device__ __forceinline__ u32x4 run(const u32x2& r) {
    return u32x4{C::lo(r[0]), C::hi(r[0]), C::lo(r[1]), C::hi(r[1])};
  }
};
template <> struct Widen8<KvFp8> : Widen8Codes<KvFp8> {};
template <> struct Widen8<KvInt8> : Widen8Codes<KvInt8> {};
template <> struct Widen8<KvInt4> {  // one word of eight nibbles
  static __device__ __forceinline__ u32x4 run(uint32_t w) {
    u32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = KvInt8::two(KvInt4::code(w, 2 * k), KvInt4::code(w, 2 * k + 1));
    return v;
  }
};

// bf16 pair of element t of two value slices (even key, odd key).
template <typename KV, typename S>
__device__ __forceinline__ uint32_t value_pair(const S& e, const S& o, int t) {
  constexpr int PER = 32 / KV::BITS;  // elements per 32-bit word
  typedef Raw<sizeof(S) < 4 ? 4 : (int)sizeof(S)> R;
  return KV::pair(R::word(e, t / PER), R::word(o, t / PER), t % PER);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Row r of QK sub-tile a holds tile key 16a + 4(r&3) + (r>>2). The logit
// accumulator of sub-tile a then gives lane (n, G) keys 16a + 4j + G
// (j = 0..3), i.e. keys 4e + G for e = 4a + j = 0..7: the same keys, in the
// same order, as the V^T operand a lane builds from value rows 4e + G.
__device__ __forceinline__ int qk_key(int a, int r) { return 16 * a + 4 * (r & 3) + (r >> 2); }

// Per-wave running state of NT query tiles. With MS (matrix-core sums) the
// row sums come from one more MFMA per tile against an all-ones operand:
// lacc holds the row's sum of the bf16-rounded weights (the weights the
// values are multiplied by) in all four of its elements, instead of the
// lane's share of the fp32 weights in l.
template <int D, int NT, bool MS = false> struct RowState {
  static constexpr int DV = D / 16;
  float mref[NT];       // reference maximum (log2 units), uniform over the row's 4 lanes
  float nbase[MS ? NT : 1];  // with MS: -mref, or 0 while mref = -inf (the exponent's offset)
  float thr[NT];        // raw-logit threshold: a logit above it calls for a higher mref
  float l[NT];          // this lane's share of the row sum (without MS)
  f32x4 lacc[MS ? NT : 1];  // row sums (with MS)
  f32x4 acc[NT][DV];    // O^T accumulators
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      mref[nt] = kNegInf;
      if constexpr (MS) nbase[nt] = 0.f;
      thr[nt] = kNegInf;
      l[nt] = 0.f;
      if constexpr (MS) lacc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < DV; ++t) acc[nt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

// One 32-key tile against NT query tiles: S^T = K Q^T on MFMA, online softmax
// with lazy rescaling, O^T += V^T P^T on MFMA. k_at(a, s) yields this lane's
// K operand of sub-tile a and k-step s, vop_at(t) its V^T operand of
// dimension block t (built on demand, so only one is live at a time),
// q_at(nt, s) its Q^T operands. `rem` counts the keys from the tile's first
// to the end of the range. With ntok tokens per (sample, group) unit (rows
// r = head*ntok + token), row r sees keys < rem - (ntok - 1) + r % ntok:
// the range ends at the last token's limit and earlier tokens stop earlier
// (ntok = 1 masks keys >= rem). Keys below `vfloor` (counted from the tile's
// first key, like rem) are seen by every row whatever its causal limit: the
// context rows that precede the decode rows in a replicated cache.
template <int D, int NT, bool MS, typename KOp, typename VOp, typename QOp>
__device__ __forceinline__ void tile_update(RowState<D, NT, MS>& st, KOp&& k_at, VOp&& vop_at,
                                            QOp&& q_at, int rem, int ntok, int vfloor,
                                            float scale_log2, int lane) {
  constexpr int KS = D / 32;
  constexpr int DV = D / 16;
  const int G = lane >> 4;
  f32x4 sacc[NT][2];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) sacc[nt][0] = sacc[nt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (MS) __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const u32x4 k0 = k_at(0, s), k1 = k_at(1, s);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const u32x4 qo = q_at(nt, s);
      sacc[nt][0] = mfma_bf16(k0, qo, sacc[nt][0]);
      sacc[nt][1] = mfma_bf16(k1, qo, sacc[nt][1]);
    }
  }
  if constexpr (MS) __builtin_amdgcn_s_setprio(0);
  // Raw logits; scale_log2 > 0, so maxima can be taken before scaling and
  // the scale folds into the exponent's multiply-add. The reference maximum
  // only has to bound the row's logits to within 2^kRescaleSlack (the same
  // reference scales its weights, sum and values): each lane compares its
  // own maximum with the threshold, and only when some lane exceeds it does
  // the wave form exact row maxima across lanes and rescale.
  float x[NT][8];  // x[nt][e]: key 4e + G
  float lmax[NT];
  bool raise_any = false;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[nt][j] = sacc[nt][0][j];
      x[nt][4 + j] = sacc[nt][1][j];
    }
    if (rem < kTileKeys + ntok - 1) {
      // The bound passes through readfirstlane (convergent), so the compiler
      // cannot hoist these compares out of the branch into every full tile.
      const int nv = __builtin_amdgcn_readfirstlane(rem) - (ntok - 1);
      const int lim = ntok == 1 ? nv
                                : max(nv + (nt * kRowsPerTile + (lane & 15)) % ntok,
                                      __builtin_amdgcn_readfirstlane(vfloor));
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (4 * e + G >= lim) x[nt][e] = kNegInf;
    }
    float m = x[nt][0];
#pragma unroll
    for (int e = 1; e < 8; ++e) m = fmaxf(m, x[nt][e]);
    lmax[nt] = m;
    raise_any |= m > st.thr[nt];
  }
  if (__any(raise_any)) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const float tmax = xor32_max(xor16_max(lmax[nt])) * scale_log2;  // exact row maximum
      // Rows that do not raise keep alpha = 1 (and never form -inf - -inf).
      const bool raise = tmax > st.mref[nt] + kRescaleSlack;
      const float alpha = raise ? exp2_fast(st.mref[nt] - tmax) : 1.f;  // 0 when mref = -inf
      if constexpr (MS)
        st.lacc[nt] *= alpha;
      else
        st.l[nt] *= alpha;
#pragma unroll
      for (int t = 0; t < DV; ++t) st.acc[nt][t] *= alpha;
      st.mref[nt] = raise ? tmax : st.mref[nt];
      if constexpr (MS) st.nbase[nt] = st.mref[nt] == kNegInf ? 0.f : -st.mref[nt];
      st.thr[nt] = (st.mref[nt] + kRescaleSlack) / scale_log2;
    }
  }
  auto weights = [&](int nt) -> u32x4 {  // bf16 P^T operand of query tile nt; adds to the sums
    // kept in the state with MS; recomputed per tile otherwise (registers)
    float nbase;
    if constexpr (MS)
      nbase = st.nbase[nt];
    else
      nbase = st.mref[nt] == kNegInf ? 0.f : -st.mref[nt];
    float pr[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pr[e] = exp2_fast(__builtin_fmaf(x[nt][e], scale_log2, nbase));
    if constexpr (!MS) {
      float psum = pr[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) psum += pr[e];
      st.l[nt] += psum;
    }
    u32x4 pb;
#pragma unroll
    for (int w = 0; w < 4; ++w) pb[w] = pack_bf16(pr[2 * w], pr[2 * w + 1]);
    if constexpr (MS) {
      constexpr uint32_t kOnes = 0x3F803F80u;  // two bf16 1.0
      st.lacc[nt] = mfma_bf16(u32x4{kOnes, kOnes, kOnes, kOnes}, pb, st.lacc[nt]);
    }
    return pb;
  };
  if constexpr (NT == 2) {
    // O^T += V^T P^T query tile by query tile, the V^T operands held. Tile
    // 1's weights do not depend on tile 0's products: they are scheduled
    // between them, so the exponentials issue while the matrix cores run
    // (sched_barrier fences the regions; group masks: 0x2 VALU, 0x8 MFMA).
    u32x4 vo[DV];
#pragma unroll
    for (int t = 0; t < DV; ++t) vo[t] = vop_at(t);
    const u32x4 pb0 = weights(0);
    __builtin_amdgcn_sched_barrier(0);
    const u32x4 pb1 = weights(1);
#pragma unroll
    for (int t = 0; t < DV; ++t) st.acc[0][t] = mfma_bf16(vo[t], pb0, st.acc[0][t]);
#pragma unroll
    for (int t = 0; t < DV; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x2, 4, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < DV; ++t) st.acc[1][t] = mfma_bf16(vo[t], pb1, st.acc[1][t]);
  } else if constexpr (NT == 1) {
    const u32x4 pb = weights(0);
    if constexpr (MS) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int t = 0; t < DV; ++t) st.acc[0][t] = mfma_bf16(vop_at(t), pb, st.acc[0][t]);
    if constexpr (MS) __builtin_amdgcn_s_setprio(0);
  } else {
    // Many query tiles: registers are short, so each V^T operand is formed
    // once and used for every tile.
    u32x4 pb[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) pb[nt] = weights(nt);
#pragma unroll
    for (int t = 0; t < DV; ++t) {
      const u32x4 v = vop_at(t);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) st.acc[nt][t] = mfma_bf16(v, pb[nt], st.acc[nt][t]);
    }
  }
}

// Q^T operands of NT query tiles. row_ptr(r) gives the bf16 row of tile row r
// (r = nt*16 + n) or nullptr when the row is padding; `sign` is XORed into
// every pair of bf16 (0x80008000 negates q for a negative softmax scale).
template <int D, int NT, typename RowPtr>
__device__ __forceinline__ void load_q(u32x4 (&qop)[NT][D / 32], RowPtr row_ptr, uint32_t sign,
                                       int lane) {
  const int n = lane & 15, G = lane >> 4;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const uint16_t* qr = row_ptr(nt * kRowsPerTile + n);
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      qop[nt][s] = qr ? load16(qr + s * 32 + G * 8) ^ sign : u32x4{0, 0, 0, 0};
  }
}

// Register path: one wave loads a whole 32-key tile, every load instruction
// reading whole consecutive rows (1 KB contiguous for d = 128 bf16):
//   K: lane l holds row RPI*e + l/CPR, 16-byte chunk l%CPR (CPR = 16-byte
//      chunks per row, RPI = 64/CPR rows per instruction); widened to bf16
//      and staged through a per-wave LDS tile to reach the MFMA operand
//      layout, whose 16 lanes each want a different row (XOR-swizzled so
//      those reads are bank-conflict free);
//   V: lane (c, G) holds row 4e + G, dims DV*c .. DV*c+DV-1 (e = 0..7), which
//      is already what its V^T operands need: formed on demand by a 16-bit
//      transpose inside the lane (widening 8-bit or 4-bit codes on the way).
// Loads go through buffer resources whose range ends at the item's last key,
// so rows past it read as zero without a branch and without a memory access.
template <int D, typename KV> struct TileRegs {
  static constexpr int KS = D / 32;
  static constexpr int DV = D / 16;
  static constexpr int RB = KV::bytes(D);  // bytes per cache row
  static constexpr int CPR = RB / 16;     // raw 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;
  static constexpr int KI = kTileKeys / RPI;
  static constexpr int BPR = D / 8;       // bf16 16-byte chunks per row in LDS
  typedef Raw<KV::bytes(DV)> VR;
  typedef typename VR::type VS;
  u32x4 kraw[KI];
  VS vrow[8];

  // Swizzled 16-byte slot of (row, bf16 chunk) in a K tile staged in LDS.
  static __device__ __forceinline__ int kslot(int row, int chunk) {
    const int swz = D == 128 ? (row & 15) : ((row >> 1) & 7);
    return row * BPR + (chunk ^ swz);
  }

  // AUX: cache policy (streamed, read-once rows by default).
  template <int AUX = kAuxStream>
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                       int key0, int lane) {
    const uint32_t koff = (uint32_t)(key0 + lane / CPR) * RB + (uint32_t)(lane % CPR) * 16;
#pragma unroll
    for (int e = 0; e < KI; ++e)
      kraw[e] = Raw<16>::load<AUX>(rk, boff(koff + (uint32_t)(e * RPI * RB)));
    const int c = lane & 15, G = lane >> 4;
    const uint32_t voff = (uint32_t)(key0 + G) * RB + (uint32_t)KV::bytes(DV * c);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      vrow[e] = VR::template load<AUX>(rv, boff(voff + (uint32_t)(4 * e * RB)));
  }
  // Write the K rows, as bf16, into this wave's LDS tile (32*d*2 bytes).
  // Lanes read each other's rows afterwards; a wave executes its LDS
  // instructions in order, and the wave barriers stop the compiler from
  // moving reads of the previous tile below these writes or reads of this
  // tile above them.
  __device__ __forceinline__ void stage_k(u32x4* kl, int lane) const {
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int e = 0; e < KI; ++e) {
      const int row = RPI * e + lane / CPR, c = lane % CPR;
      const u32x4& w = kraw[e];
      if constexpr (KV::BITS == 16) {
        *(lds_u32x4*)(kl + kslot(row, c)) = w;
      } else if constexpr (KV::BITS == 8) {
        // 16 codes: bf16 chunks 2c and 2c + 1 of the row.
        *(lds_u32x4*)(kl + kslot(row, 2 * c)) = Widen8<KV>::run(u32x2{w[0], w[1]});
        *(lds_u32x4*)(kl + kslot(row, 2 * c + 1)) = Widen8<KV>::run(u32x2{w[2], w[3]});
      } else {
        // 32 codes: bf16 chunks 4c .. 4c + 3 of the row.
#pragma unroll
        for (int k = 0; k < 4; ++k)
          *(lds_u32x4*)(kl + kslot(row, 4 * c + k)) = Widen8<KV>::run(w[k]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // K operand of sub-tile a, k-step s: row qk_key(a, n), dims 32s + 8G .. +7.
  static __device__ __forceinline__ u32x4 kop(const u32x4* kl, int a, int s, int lane) {
    return *(const lds_u32x4*)(kl + kslot(qk_key(a, lane & 15), 4 * s + (lane >> 4)));
  }
  // Zero the value rows of keys >= nvalid (rows past a sample's length may
  // hold anything; their weight is 0 but 0 * NaN is not). Zero bytes are the
  // value 0 in every cache type.
  __device__ __forceinline__ void mask_v(int nvalid, int lane) {
    const int G = lane >> 4;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (4 * e + G >= nvalid) vrow[e] = VR::zero();
  }
  // V^T operand of dimension block t: keys 4(2w) + G, 4(2w+1) + G in word w.
  __device__ __forceinline__ u32x4 vop(int t) const {
    u32x4 v;
#pragma unroll
    for (int w = 0; w < 4; ++w) v[w] = value_pair<KV>(vrow[2 * w], vrow[2 * w + 1], t);
    return v;
  }
};

// Buffer resource over `rows` cache rows of `row_bytes` starting at `base`
// (raw, stride 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const uint8_t* base, int rows,
                                                             int row_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), (short)0, rows * row_bytes,
                                           0x00020000);
}

// Row totals of the per-lane sums (the four lanes of a row share the row).
template <int D, int NT, bool MS>
__device__ __forceinline__ void finish_sums(RowState<D, NT, MS>& st) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    if constexpr (MS)
      st.l[nt] = st.lacc[nt][0];
    else
      st.l[nt] = xor32_sum(xor16_sum(st.l[nt]));
  }
}

// Write the wave's partials of rows row0 + nt*16 + n < nrows: lane (n, G)
// stores dims [4*DV*G, 4*DV*G + 4*DV) of its row (contiguous), lane G = 0
// the row's (m, l).
template <int D, int NT>
__device__ __forceinline__ void store_partials(RowState<D, NT>& st, int nrows, float* acc_out,
                                               float2* ml_out, int lane) {
  constexpr int DV = D / 16;
  const int n = lane & 15, G = lane >> 4;
  finish_sums(st);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int row = nt * kRowsPerTile + n;
    if (row < nrows) {
      float* dst = acc_out + (size_t)row * D + 4 * DV * G;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int t4 = 0; t4 < DV; t4 += 4)
          *reinterpret_cast<f32x4*>(dst + DV * j + t4) =
              f32x4{st.acc[nt][t4][j], st.acc[nt][t4 + 1][j], st.acc[nt][t4 + 2][j],
                    st.acc[nt][t4 + 3][j]};
      if (G == 0) ml_out[row] = float2{st.mref[nt], st.l[nt]};
    }
  }
}

// One wave streams the 32-key tiles starting at keys k0, k0 + stride,
// k0 + 2*stride, ... below k1 of one cache segment (buffer resources rk/rv
// over its rows) through tile_update, double-buffered: the loads of the
// next tile are issued before the current one is consumed, so a tile is
// always in flight. The caller has already issued the loads of the first tile
// into A (before anything else, so that they overlap the set-up). The waves
// that share a segment start at neighbouring tiles, so together they sweep
// one window of it. qw: this wave's Q^T operands in LDS, [NT][d/32][64
// lanes]; kl: this wave's LDS K tile (32*d*2 bytes). kend: the end of the
// sequence the tokens' causal limits count from (ntok tokens per unit; k1
// when ntok = 1); keys below vis0 are seen by every token.
template <int D, int NT, typename KV, int AUX = kAuxStream>
__device__ __forceinline__ void stream_keys(RowState<D, NT>& st, const u32x4* qw, u32x4* kl,
                                            __amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                            TileRegs<D, KV>& A, int k0, int k1, int kend, int stride,
                                            int ntok, int vis0, float scale_log2, int lane) {
  constexpr int KS = D / 32;
  if (k0 >= k1) return;
  // Volatile: a real LDS read at each use, not a register copy kept alive
  // across the loop (which would cost 16 registers per query tile).
  auto q_at = [&](int nt, int s) -> u32x4 {
    return *(volatile const lds_u32x4*)(qw + (nt * KS + s) * 64 + lane);
  };
  auto k_at = [&](int a, int s) { return TileRegs<D, KV>::kop(kl, a, s, lane); };
  TileRegs<D, KV> B;
  // Prefetches are unconditional: past the resource range the buffer load
  // returns zeros without a memory access, and a fixed count of loads in
  // flight lets each wait cover only the tile being consumed.
  for (int key = k0;; key += 2 * stride) {
    const int key1 = key + stride;
    B.template load<AUX>(rk, rv, key1, lane);
    const int nv0 = min(kTileKeys, k1 - key);
    if (nv0 < kTileKeys) A.mask_v(nv0, lane);
    A.stage_k(kl, lane);
    tile_update<D, NT>(st, k_at, [&](int t) { return A.vop(t); }, q_at, kend - key, ntok,
                       vis0 - key, scale_log2, lane);
    if (key1 >= k1) break;
    const int key2 = key1 + stride;
    A.template load<AUX>(rk, rv, key2, lane);
    const int nv1 = min(kTileKeys, k1 - key1);
    if (nv1 < kTileKeys) B.mask_v(nv1, lane);
    B.stage_k(kl, lane);
    tile_update<D, NT>(st, k_at, [&](int t) { return B.vop(t); }, q_at, kend - key1, ntok,
                       vis0 - key1, scale_log2, lane);
    if (key2 >= k1) break;
  }
}

// Stage this wave's Q^T operands of NT query tiles in its LDS slice qw.
// row_ptr(r) gives the bf16 row of tile row r (r = nt*16 + n) or nullptr
// for padding rows.
template <int D, int NT, typename RowPtr>
__device__ __forceinline__ void stage_q(u32x4* qw, RowPtr row_ptr, uint32_t sign, int lane) {
  constexpr int KS = D / 32;
  u32x4 qop[NT][KS];
  load_q<D, NT>(qop, row_ptr, sign, lane);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      *(volatile lds_u32x4*)(qw + (nt * KS + s) * 64 + lane) = qop[nt][s];
}

// Softmax scale of group gam's units in log2 units, the key scale folded in
// (logit = scale * k_scale * q . code values).
__device__ __forceinline__ float unit_scale_log2(const PartialsParams& P, int gam) {
  return P.k_scale ? P.scale_log2 * P.k_scale[gam] : P.scale_log2;
}

constexpr int cmax(int a, int b) { return a > b ? a : b; }

__device__ __forceinline__ int clamp_len(const int32_t* lens, int i, int m_d_max) {
  const int raw = lens ? lens[i] : 0;
  return raw < 0 ? 0 : (raw > m_d_max ? m_d_max : raw);
}

// ---------------------------------------------------------------------------
// Decode part (and the replicated ablation): work-group (sample i, group gam,
// key chunk s) over the sample's own cache rows [s*dec_keys,
// min((s+1)*dec_keys, len)). Its four waves take interleaved tiles and each
// writes its own partial of the p query rows of group gam (partial slot
// (chunk, wave)); a wave without keys writes the empty partial
// (m = -inf, l = 0, acc = 0).
template <int D, int NT, typename KV>
__device__ void decode_block(const PartialsParams& P, int blk, int wave, int lane, u32x4* qw,
                             u32x4* kl) {
  constexpr int RB = KV::bytes(D);
  const int s = blk % P.S_d;
  const int ig = blk / P.S_d;
  const int gam = ig % P.g, i = ig / P.g;
  const int kbeg = s * P.dec_keys;
  const int kcap = min(P.dec_rows, kbeg + P.dec_keys);  // the chunk within the cache capacity
  const size_t cache = (size_t)(i * P.g + gam) * P.dec_rows * RB;
  const __amdgpu_buffer_rsrc_t rk = rows_rsrc(P.Kd + cache, kcap, RB);
  const __amdgpu_buffer_rsrc_t rv = rows_rsrc(P.Vd + cache, kcap, RB);
  const int k0 = kbeg + wave * kTileKeys;
  TileRegs<D, KV> A;
  A.load(rk, rv, k0, lane);  // first tile in flight before the length is known
  const int total = P.len_offset + clamp_len(P.lens, i, P.m_d_max);
  const int k1 = min(total, kcap);
  // Now that the length is known, later loads (the prefetch of each wave's
  // next tile included) stop at the sample's last valid row: past it they
  // return zeros without touching memory, so the masked tail is never read.
  const __amdgpu_buffer_rsrc_t rk1 = rows_rsrc(P.Kd + cache, k1, RB);
  const __amdgpu_buffer_rsrc_t rv1 = rows_rsrc(P.Vd + cache, k1, RB);
  const uint16_t* qbase = P.q + ((size_t)i * P.h + (size_t)gam * P.p) * D;
  const int p = P.p;
  stage_q<D, NT>(qw, [&](int r) -> const uint16_t* { return r < p ? qbase + (size_t)r * D : nullptr; },
                 P.q_sign, lane);
  RowState<D, NT> st;
  st.init();
  // Keys [k0, k1) of this chunk; the causal limits of the tokens count from
  // the end of the sequence (total), which may lie in a later chunk.
  stream_keys<D, NT, KV>(st, qw, kl, rk1, rv1, A, k0, k1, total, kWaves * kTileKeys, P.ntok,
                         P.len_offset, unit_scale_log2(P, gam), lane);
  const size_t prow = ((size_t)blk * kWaves + wave) * P.p;
  store_partials<D, NT>(st, p, P.dec_acc + prow * D, P.dec_ml + prow, lane);
}

// Merge the four waves' states of the same NT*16 rows through LDS, in wave
// order (so the result is deterministic): afterwards row r's merged partial
// is acc_s[r*LD ..], m_s[r], l_s[r] (LD = d + 4), visible to every thread.
template <int D, int NT>
__device__ __forceinline__ void merge_waves(RowState<D, NT>& st, float* lds, int wave, int lane) {
  constexpr int DV = D / 16;
  constexpr int LD = D + 4;  // padded LDS row
  constexpr int ROWS = NT * kRowsPerTile;
  float* acc_s = lds;
  float* m_s = lds + ROWS * LD;
  float* l_s = m_s + ROWS;
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
}

// Merge the waves' states and write rows < nrows of the merged partial to
// acc_out / ml_out.
template <int D, int NT>
__device__ __forceinline__ void merge_waves_and_store(RowState<D, NT>& st, float* lds, int nrows,
                                                      float* acc_out, float2* ml_out, int wave,
                                                      int lane) {
  constexpr int LD = D + 4;
  constexpr int ROWS = NT * kRowsPerTile;
  merge_waves<D, NT>(st, lds, wave, lane);
  const float* acc_s = lds;
  const float* m_s = lds + ROWS * LD;
  const float* l_s = m_s + ROWS;
  constexpr int V4 = D / 4;
  for (int idx = threadIdx.x; idx < nrows * V4; idx += kThreads) {
    const int row = idx / V4, c = idx % V4;
    *reinterpret_cast<f32x4*>(acc_out + (size_t)row * D + 4 * c) =
        *reinterpret_cast<const f32x4*>(acc_s + row * LD + 4 * c);
  }
  for (int row = threadIdx.x; row < nrows; row += kThreads) ml_out[row] = float2{m_s[row], l_s[row]};
}

template <int D, int NT> struct MergeLds {
  static constexpr int bytes = (NT * kRowsPerTile * (D + 4) + 2 * NT * kRowsPerTile) * 4;
};

// Context part, few query rows per group (M = b*p <= 64): work-group
// (group gam, split s) of S_c per group. The 4*S_c waves of a group take the
// group's 32-key tiles round robin (wave w of split s: tiles 4s+w,
// 4s+w+4*S_c, ...), so they sweep K_c/V_c together and each tile is read
// once, straight into the operands that serve all M query rows. The four
// waves' states merge in LDS into the split's partial.
template <int D, int NT, typename KV>
__device__ void ctx_small_block(const PartialsParams& P, int blk, int wave, int lane, u32x4* qw,
                                u32x4* kl, float* merge_lds) {
  constexpr int RB = KV::bytes(D);
  const int s = blk % P.S_c, gam = blk / P.S_c;
  const size_t cache = (size_t)gam * P.m_c * RB;
  const __amdgpu_buffer_rsrc_t rk = rows_rsrc(P.Kc + cache, P.m_c, RB);
  const __amdgpu_buffer_rsrc_t rv = rows_rsrc(P.Vc + cache, P.m_c, RB);
  const int k0 = (s * kWaves + wave) * kTileKeys;
  TileRegs<D, KV> A;
  A.load(rk, rv, k0, lane);  // first tile in flight while Q is staged
  const int M = P.M, p = P.p, h = P.h;
  const uint16_t* q = P.q;
  stage_q<D, NT>(qw, [&](int r) -> const uint16_t* {
    if (r >= M) return nullptr;
    const int i = r / p, jp = r - i * p;
    return q + ((size_t)i * h + (size_t)gam * p + jp) * D;
  }, P.q_sign, lane);
  RowState<D, NT> st;
  st.init();
  stream_keys<D, NT, KV>(st, qw, kl, rk, rv, A, k0, P.m_c, P.m_c, P.S_c * kWaves * kTileKeys, 1,
                         0, unit_scale_log2(P, gam), lane);
  const size_t prow = (size_t)blk * P.M;
  __syncthreads();  // the merge buffer overlays the waves' K tiles
  merge_waves_and_store<D, NT>(st, merge_lds, M, P.ctx_acc + prow * D, P.ctx_ml + prow, wave, lane);
}

// Standard attention, the other side of the workload-based switch (FAQ on
// caveats: splitting the attention costs parallelism on small workloads, so
// they run the plain computation): work-group (sample i, group gam) streams
// the whole sequence of the unit, the group's context rows and then the
// sample's decode rows, as one softmax (Section 3.3, Eq. 1-2). The context
// is read once per sample instead of once per group, so this only pays where
// launches and latency, not bytes, set the time. The four waves take
// interleaved tiles of each segment, merge in LDS and write the normalized
// output rows (times the group's value scale) directly: one launch, no
// partials, no combine. The unit with gam = 0 checks the sample's length and
// the unit with i = 0 its group's scales.
template <int D, int NT, typename KV>
__device__ void standard_block(const PartialsParams& P, int blk, int wave, int lane, u32x4* qw,
                               u32x4* kl, float* merge_lds) {
  constexpr int RB = KV::bytes(D);
  constexpr int LD = D + 4;
  constexpr int ROWS = NT * kRowsPerTile;
  const int gam = blk % P.g, i = blk / P.g;
  const __amdgpu_buffer_rsrc_t rkc = rows_rsrc(P.Kc + (size_t)gam * P.m_c * RB, P.m_c, RB);
  const __amdgpu_buffer_rsrc_t rvc = rows_rsrc(P.Vc + (size_t)gam * P.m_c * RB, P.m_c, RB);
  const int k0 = wave * kTileKeys;
  constexpr int stride = kWaves * kTileKeys;
  TileRegs<D, KV> A;
  // The context rows are read once per sample here: loaded with the default
  // cache policy, so that the group's other samples may find them cached.
  A.template load<0>(rkc, rvc, k0, lane);  // first context tile in flight during the set-up
  const int p = P.p;
  const uint16_t* qbase = P.q + ((size_t)i * P.h + (size_t)gam * p) * D;
  stage_q<D, NT>(qw, [&](int r) -> const uint16_t* { return r < p ? qbase + (size_t)r * D : nullptr; },
                 P.q_sign, lane);
  const float sl2 = unit_scale_log2(P, gam);
  RowState<D, NT> st;
  st.init();
  // Context rows: visible to every token (a causal limit only applies among
  // the decode rows).
  stream_keys<D, NT, KV, 0>(st, qw, kl, rkc, rvc, A, k0, P.m_c, P.m_c, stride, 1, 0, sl2, lane);
  const int len = clamp_len(P.lens, i, P.m_d_max);
  if (len > 0) {  // wave-uniform
    const size_t cache = (size_t)(i * P.g + gam) * P.m_d_max * RB;
    const __amdgpu_buffer_rsrc_t rkd = rows_rsrc(P.Kd + cache, len, RB);
    const __amdgpu_buffer_rsrc_t rvd = rows_rsrc(P.Vd + cache, len, RB);
    A.load(rkd, rvd, k0, lane);
    stream_keys<D, NT, KV>(st, qw, kl, rkd, rvd, A, k0, len, len, stride, P.ntok, 0, sl2, lane);
  }
  __syncthreads();  // the merge buffer overlays the waves' K tiles
  merge_waves<D, NT>(st, merge_lds, wave, lane);
  const float vs = P.v_scale ? P.v_scale[gam] : 1.f;
  const float* acc_s = merge_lds;
  const float* l_s = merge_lds + ROWS * LD + ROWS;
  float* out = P.out + ((size_t)i * P.h + (size_t)gam * p) * D;
  constexpr int V4 = D / 4;
  for (int idx = threadIdx.x; idx < p * V4; idx += kThreads) {
    const int row = idx / V4, c = idx % V4;
    const float inv = vs / l_s[row];
    *reinterpret_cast<f32x4*>(out + (size_t)row * D + 4 * c) =
        *reinterpret_cast<const f32x4*>(acc_s + row * LD + 4 * c) * inv;
  }
  if (threadIdx.x == 0) {
    int flags = 0;
    if (gam == 0 && P.lens) {
      const int raw = P.lens[i];
      if (raw < 0 || raw > P.m_d_max) flags |= kStatusLens;
    }
    if (i == 0) {
      const float ks = P.k_scale ? P.k_scale[gam] : 1.f;
      if (!(ks >= __FLT_MIN__ && ks <= __FLT_MAX__ && vs >= __FLT_MIN__ && vs <= __FLT_MAX__))
        flags |= kStatusScale;
    }
    if (flags) atomicOr(P.status, flags);
  }
}

template <int D, int NT, typename KV>
__global__ __launch_bounds__(kThreads) void standard_kernel(PartialsParams P) {
  constexpr int QSLOTS = kWaves * NT * (D / 32) * 64;
  constexpr int KSLOTS = kWaves * kTileKeys * D / 8;
  constexpr int MERGE = (MergeLds<D, NT>::bytes + 15) / 16;  // overlays the K tiles
  __shared__ __attribute__((aligned(16))) u32x4 lds[QSLOTS + cmax(KSLOTS, MERGE)];
  const int lane = threadIdx.x & 63, wave = wave_id();
  u32x4* qw = lds + wave * NT * (D / 32) * 64;
  u32x4* kl = lds + QSLOTS + wave * (kTileKeys * D / 8);
  if ((int)blockIdx.x < P.b * P.g)
    standard_block<D, NT, KV>(P, blockIdx.x, wave, lane, qw, kl,
                              reinterpret_cast<float*>(lds + QSLOTS));
}


// Context part, many query rows per group: work-group (group gam, key split
// s, row block rb) of 128 query rows, eight waves with one 16-row query
// tile each, two work-groups per CU (four waves per SIMD, so one wave's
// softmax arithmetic overlaps another's matrix products and waits).
// Each 32-key tile of Kc/Vc is loaded from HBM once per work-group into LDS,
// already in MFMA operand order (the V^T transpose is done once, on the way
// in), and all eight waves read it. Each wave stages one eighth of a tile:
// one K operand (d = 128; the first four waves for d = 64) and one 32-bit
// word of half of the V^T operands, widening 8-bit or 4-bit codes to bf16 on
// the way. Tiles are double-buffered in LDS with one barrier per tile, and
// fetched three tiles ahead into three rotating register sets. Q^T operands stay in registers. Row blocks of one key
// chunk are scheduled on the same XCD so that they share its L2.
template <int D, typename KV>
__device__ __forceinline__ void ctx_large_body(const PartialsParams& P) {
  constexpr int KS = D / 32;
  constexpr int DV = D / 16;
  constexpr int RB = KV::bytes(D);  // bytes per cache row
  constexpr int KOPS = 2 * KS;    // K operands per tile
  constexpr int OPS = KOPS + DV;  // operands per tile (16 B per lane each)
  constexpr int HW = DV / 2;      // V^T operands one wave stages a word of
  typedef Raw<KV::bytes(8)> KR;   // a lane's 8 elements of its K operand
  typedef Raw<KV::bytes(HW)> VR;  // a lane's HW elements of a value row
  typedef typename VR::type VH;
  __shared__ __attribute__((aligned(16))) u32x4 lds[2 * OPS * 64];
  const int blk = xcd_logical(blockIdx.x, P.g * P.S_c, P.ctx_row_blocks);
  const int rb = blk % P.ctx_row_blocks;
  const int sg = blk / P.ctx_row_blocks;
  const int s = sg % P.S_c, gam = sg / P.S_c;
  const int k0 = s * P.ctx_keys;
  const int nkeys = min(P.m_c, k0 + P.ctx_keys) - k0;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int r = lane & 15, G = lane >> 4;
  // Buffer resources over the chunk's keys [k0, k0 + nkeys): rows past it
  // load as zero with no memory access and no branch. Offsets count from k0.
  const size_t chunk = ((size_t)gam * P.m_c + k0) * RB;
  const __amdgpu_buffer_rsrc_t rk = rows_rsrc(P.Kc + chunk, nkeys, RB);
  const __amdgpu_buffer_rsrc_t rv = rows_rsrc(P.Vc + chunk, nkeys, RB);
  const float scale_log2 = unit_scale_log2(P, gam);
  const int M = P.M, p = P.p, h = P.h;
  const int row0 = rb * kLargeRowsPerBlock + wave * kRowsPerTile;
  auto slot = [&](int buf, int op) -> u32x4* { return lds + (buf * OPS + op) * 64; };
  const bool has_k = wave < KOPS;              // wave-uniform
  const int ka = wave / KS, kss = wave % KS;   // the K operand this wave stages
  const int vw = wave & 3, vh = wave >> 2;     // its V^T word and operand half

  // Registers of a tile in flight: this wave's K operand and two value-row halves.
  struct Stage {
    typename KR::type k;
    VH v[2];
  };
  auto fetch = [&](Stage& g, int key0) {  // keys past the chunk load as zero
    if (has_k)
      g.k = KR::load(rk, boff((uint32_t)(key0 + qk_key(ka, r)) * RB +
                              (uint32_t)KV::bytes(kss * 32 + G * 8)));
#pragma unroll
    for (int c = 0; c < 2; ++c)
      g.v[c] = VR::load(rv, boff((uint32_t)(key0 + 4 * (2 * vw + c) + G) * RB +
                                 (uint32_t)KV::bytes(DV * r + vh * HW)));
  };
  auto stage = [&](const Stage& g, int buf) {
    if (has_k) slot(buf, wave)[lane] = Widen8<KV>::run(g.k);
    // word vw of V^T operand vh*HW + t = keys 4(2vw) + G, 4(2vw+1) + G at dim DV*r + vh*HW + t
#pragma unroll
    for (int t = 0; t < HW; ++t)
      reinterpret_cast<uint32_t*>(slot(buf, KOPS + vh * HW + t) + lane)[vw] =
          value_pair<KV>(g.v[0], g.v[1], t);
  };

  // Q first, then the first two tiles: the wait for the first tile then also
  // covers Q, so no wait inside the loop reaches past the set in flight.
  u32x4 qop[1][KS];
  load_q<D, 1>(qop, [&](int rr) -> const uint16_t* {
    const int row = row0 + rr;
    if (row >= M) return nullptr;
    const int i = row / p, jp = row - i * p;
    return P.q + ((size_t)i * h + (size_t)gam * p + jp) * D;
  }, P.q_sign, lane);
  constexpr int T = kTileKeys;
  Stage S0, S1, S2;
  fetch(S0, 0);
  fetch(S1, T);
  fetch(S2, 2 * T);
  RowState<D, 1, true> st;
  st.init();
  const bool rows = row0 < M;  // wave-uniform: waves past the last row only stage
  stage(S0, 0);
  __syncthreads();
  // Tile `key` (in LDS buffer buf) is consumed while the next two tiles are
  // in flight in two register sets and the one after them is issued into
  // the third (the set tile `key` came from); fetches past the chunk are
  // unconditional (they read zeros), so every wait covers exactly one set.
  // The loop runs six tiles per turn while a seventh follows (a single exit
  // at the bottom keeps the waits exact); the last one to six tiles are the
  // tail.
  auto step = [&](int key, int buf, Stage& spare, Stage& next, bool stage_next) {
    fetch(spare, key + 3 * T);
    if (rows)
      tile_update<D, 1>(st, [&](int a, int ss) { return slot(buf, a * KS + ss)[lane]; },
                        [&](int t) { return slot(buf, KOPS + t)[lane]; },
                        [&](int, int ss) { return qop[0][ss]; }, nkeys - key, 1, 0,
                        scale_log2, lane);
    if (stage_next) {
      // The other buffer was last read in the previous step, before the
      // barrier that ended it.
      stage(next, buf ^ 1);
      __syncthreads();
    }
  };
  int key = 0;
  for (; key + 6 * T < nkeys; key += 6 * T) {
    step(key, 0, S0, S1, true);
    step(key + T, 1, S1, S2, true);
    step(key + 2 * T, 0, S2, S0, true);
    step(key + 3 * T, 1, S0, S1, true);
    step(key + 4 * T, 0, S1, S2, true);
    step(key + 5 * T, 1, S2, S0, true);
  }
  step(key, 0, S0, S1, key + T < nkeys);
  if (key + T < nkeys) step(key + T, 1, S1, S2, key + 2 * T < nkeys);
  if (key + 2 * T < nkeys) step(key + 2 * T, 0, S2, S0, key + 3 * T < nkeys);
  if (key + 3 * T < nkeys) step(key + 3 * T, 1, S0, S1, key + 4 * T < nkeys);
  if (key + 4 * T < nkeys) step(key + 4 * T, 0, S1, S2, key + 5 * T < nkeys);
  if (key + 5 * T < nkeys) step(key + 5 * T, 1, S2, S0, false);

  finish_sums(st);
  const int row = row0 + r;
  if (row < M) {
    const size_t prow = ((size_t)gam * P.S_c + s) * P.M + row;
    float* dst = P.ctx_acc + prow * D + 4 * DV * G;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t4 = 0; t4 < DV; t4 += 4)
        *reinterpret_cast<f32x4*>(dst + DV * j + t4) =
            f32x4{st.acc[0][t4][j], st.acc[0][t4 + 1][j], st.acc[0][t4 + 2][j],
                  st.acc[0][t4 + 3][j]};
    if (G == 0) P.ctx_ml[prow] = float2{st.mref[0], st.l[0]};
  }
}

template <int D, typename KV>
__global__ __launch_bounds__(kLargeThreads) __attribute__((amdgpu_waves_per_eu(4))) void
ctx_large_kernel(PartialsParams P) {
  ctx_large_body<D, KV>(P);
}


// ---------------------------------------------------------------------------
// Context part, many query rows per group, d = 128 (any cache type), on
// v_mfma_f32_32x32x16_bf16 (lane l, j = l % 32, h = l / 32):
//   A (32 x 16): lane holds A[j][8h .. 8h+7]
//   B (16 x 32): lane holds B[8h .. 8h+7][j]
//   C (32 x 32): element v of lane l is C[8(v/4) + 4h + v%4][j]
// Work-group (group gam, key split s, row block rb) of NW waves, each with
// 32 query rows. Logits are computed transposed, S^T = K Q^T (A: 32 keys of
// K, B: Q^T from registers), so a lane's 16 accumulator elements are logits
// of its own query row j, keys 8(v/4) + 4h + v%4 of the 32-key block. The
// value product is O^T += V^T P^T over two 16-key steps: k-step s uses the
// lane's elements v = 8s .. 8s+7 as its P^T operand, i.e. MFMA k-slot 8h + e
// stands for key 16s + 8(e/4) + 4h + e%4, and the V^T operand of dims
// 32t .. 32t+31 holds the same keys, read from key-major value rows with two
// transposing LDS reads (ds_read_b64_tr_b16: in each group of 16 lanes,
// lane i receives element i % 4 of the 4-element chunks that lanes i/4,
// 4 + i/4, 8 + i/4, 12 + i/4 address; lane i' of group q addresses key
// 16s + 8r + 4(q/2) + i'/4, dims 32t + 16(q%2) + 4(i'%4), read r = 0, 1).
// Keys stream in stages of SK (64 or 128: two or four 32-key blocks)
// through a ring of NB stage buffers in LDS of bf16 rows. bf16 caches fill
// them straight from memory by buffer loads to LDS (lane l's 16 bytes land
// at the instruction's base + 16 l, so the lane chooses which chunk of which
// row to fetch); code caches load a stage into registers a stage ahead and
// write it widened (stage_get / stage_put). Rows are padded in LDS, key
// rows to 272 bytes and value rows to 288, which keeps both kinds of operand
// reads free of bank conflicts (16 key rows of one read start 16 bytes
// apart in the banks, the 4 value rows of one transposing read 32 bytes
// apart) while every read address stays a per-lane base plus a constant;
// the lanes that fill padding load from beyond the buffer's range, which
// writes zeros without a memory access. One barrier per stage hands a
// filled buffer to every wave and releases the oldest for refilling.
namespace wide {
constexpr int D = 128;
constexpr int RB = D * 2;             // bytes per bf16 row
constexpr int KSTEPS = D / 16;        // k-steps of the logits
constexpr int DB = D / 32;            // 32-dim blocks of the output
constexpr int KROW = RB + 16;         // padded key row in LDS
constexpr int VROW = RB + 32;         // padded value row in LDS
constexpr int KSLOTS = KROW / 16;     // 17 sixteen-byte slots per key row
constexpr int VSLOTS = VROW / 16;     // 18 per value row
constexpr uint32_t kBeyond = 0x80000000u;  // a byte offset past any cache chunk
}  // namespace wide

typedef __attribute__((address_space(3))) void lds_void;
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short v4i16 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Transposing LDS read (ds_read_b64_tr_b16) at LDS byte address addr + OFF,
// issued as inline assembly: the compiler places a wait for every
// buffer-to-LDS load in flight before its own form of this read (it cannot
// tell that those loads fill the other stage buffer), which would expose the
// next stage's load latency once per stage. The caller orders the read after
// the stage's own loads (wait and barrier) and waits for its data with
// lds_wait_tr before using it.
template <int OFF>
__device__ __forceinline__ u32x2 ds_tr16(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
  return r;
}
// Waits until every LDS read issued so far has returned; the registers pass
// through the statement, so no use of them can move above the wait.
__device__ __forceinline__ void lds_wait_tr(u32x2 (&w)[16]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(w[4]), "+v"(w[5]),
                 "+v"(w[6]), "+v"(w[7]), "+v"(w[8]), "+v"(w[9]), "+v"(w[10]), "+v"(w[11]),
                 "+v"(w[12]), "+v"(w[13]), "+v"(w[14]), "+v"(w[15])
               :
               : "memory");
}
// Key operand read (ds_read_b128) at LDS byte address addr + OFF, by inline
// assembly like ds_tr16 (so that its wait can be placed by the caller, with
// lds_wait_k, after the value products it overlaps).
template <int OFF>
__device__ __forceinline__ u32x4 ds_b128(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
  return r;
}
__device__ __forceinline__ void lds_wait_k(u32x4 (&w)[8]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(w[4]), "+v"(w[5]),
                 "+v"(w[6]), "+v"(w[7])
               :
               : "memory");
}
// The eight key operands (k-steps 0..7) of one 32-key block of key rows
// padded to 272 bytes: read ks at 32 ks bytes from the lane's base.
__device__ __forceinline__ void read_k_block(uint32_t a, u32x4 (&w)[8]) {
  w[0] = ds_b128<0>(a); w[1] = ds_b128<32>(a); w[2] = ds_b128<64>(a); w[3] = ds_b128<96>(a);
  w[4] = ds_b128<128>(a); w[5] = ds_b128<160>(a); w[6] = ds_b128<192>(a); w[7] = ds_b128<224>(a);
}
// The sixteen transposing reads of one 32-key block's V^T operands: read
// (ss, t, r) of k-step ss, dims 32t .. 32t+31, half r, into w[8 ss + 2 t + r].
template <int VROW>
__device__ __forceinline__ void read_vt_block(uint32_t a, u32x2 (&w)[16]) {
#define BIFATTN_TR(ss, t, r) w[8 * (ss) + 2 * (t) + (r)] = ds_tr16<(16 * (ss) + 8 * (r)) * VROW + 64 * (t)>(a)
  BIFATTN_TR(0, 0, 0); BIFATTN_TR(0, 0, 1); BIFATTN_TR(0, 1, 0); BIFATTN_TR(0, 1, 1);
  BIFATTN_TR(0, 2, 0); BIFATTN_TR(0, 2, 1); BIFATTN_TR(0, 3, 0); BIFATTN_TR(0, 3, 1);
  BIFATTN_TR(1, 0, 0); BIFATTN_TR(1, 0, 1); BIFATTN_TR(1, 1, 0); BIFATTN_TR(1, 1, 1);
  BIFATTN_TR(1, 2, 0); BIFATTN_TR(1, 2, 1); BIFATTN_TR(1, 3, 0); BIFATTN_TR(1, 3, 1);
#undef BIFATTN_TR
}

template <int NW, int NB, int SK, typename KV>
__device__ __forceinline__ void ctx_wide_body(const PartialsParams& P) {
  using wide::D;
  using wide::RB;
  using wide::KSTEPS;
  using wide::DB;
  using wide::KROW;
  using wide::VROW;
  using wide::KSLOTS;
  using wide::VSLOTS;
  using wide::kBeyond;
  constexpr int KAREA = SK * KROW;
  constexpr int VAREA = SK * VROW;
  constexpr int STAGE = KAREA + VAREA;
  constexpr int LOADS = STAGE / 1024;
  constexpr int LPW = (LOADS + NW - 1) / NW;   // loads per wave per stage (the last ones fewer)
  constexpr int FULL = LOADS - (LPW - 1) * NW;  // waves with LPW loads; the rest have LPW - 1
  static_assert(STAGE % 1024 == 0 && KAREA % 1024 == 0, "stage areas are whole loads");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[NB * STAGE];
  const int blk = xcd_logical(blockIdx.x, P.g * P.S_c, P.ctx_row_blocks);
  const int rb = blk % P.ctx_row_blocks;
  const int sg = blk / P.ctx_row_blocks;
  const int s = sg % P.S_c, gam = sg / P.S_c;
  const int k0 = s * P.ctx_keys;
  const int nkeys = min(P.m_c, k0 + P.ctx_keys) - k0;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int j = lane & 31, h = lane >> 5;
  // Caches of bf16 load straight into LDS; code caches are staged through
  // registers and widened to bf16 on the way (same LDS layout).
  constexpr bool kDirect = KV::BITS == 16;
  static_assert(kDirect || NB == 2, "code caches use two stage buffers");
  constexpr int CRB = KV::bytes(D);  // bytes per cache row in memory
  const uint8_t* kchunk = P.Kc + ((size_t)gam * P.m_c + k0) * CRB;
  const uint8_t* vchunk = P.Vc + ((size_t)gam * P.m_c + k0) * CRB;
  const float sl2 = unit_scale_log2(P, gam);
  const int M = P.M, p = P.p;
  const int row0 = rb * (32 * NW) + wave * 32;
  const int nload = wave < FULL ? LPW : LPW - 1;  // wave-uniform

  // Byte offset, from a stage's first key, of the 16 bytes this lane loads
  // in its u-th load of every stage (load i = wave + NW u fills LDS bytes
  // [1024 i, 1024 i + 1024) of the stage: key rows, then value rows).
  uint32_t loff[LPW];
#pragma unroll
  for (int u = 0; u < LPW; ++u) {
    const int slot = 64 * (wave + NW * u) + lane;  // 16-byte slot of the stage
    const bool is_v = slot >= KAREA / 16;
    const int vs = slot - KAREA / 16;
    const int row = is_v ? vs / VSLOTS : slot / KSLOTS;
    const int c = is_v ? vs % VSLOTS : slot % KSLOTS;
    loff[u] = c < 16 ? (uint32_t)(row * RB + c * 16) : kBeyond;
  }
  auto fetch = [&](int key0, int buf) {
    const int rows = nkeys - key0;  // rows from the stage's first key to the chunk's end
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(kchunk + (size_t)key0 * CRB, rows, CRB);
    const __amdgpu_buffer_rsrc_t rv = rows_rsrc(vchunk + (size_t)key0 * CRB, rows, CRB);
#pragma unroll
    for (int u = 0; u < LPW; ++u) {
      if (u < nload) {
        const int i = wave + NW * u;  // wave-uniform
        lds_void* dst = (lds_void*)(lds + buf * STAGE + i * 1024);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(i < KAREA / 1024 ? rk : rv, dst, 16,
                                                 boff(loff[u]), 0, 0, 0);
      }
    }
  };
  // This wave's loads of stage st are complete once at most the loads of
  // the one stage issued after it are in flight (or none, at the end).
  auto wait_stage = [&](bool last) {
    if (last || NB == 2)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (nload == LPW)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPW - 1) : "memory");
  };

  // Q^T operands: k-step ks holds dims 16ks + 8h .. +7 of query row j.
  // Rows past M load row M - 1 and are zeroed afterwards, so that the eight
  // loads issue back to back (a load under a per-lane condition waits for
  // its data before the next one issues).
  u32x4 qop[KSTEPS];
  {
    const int row = row0 + j;
    const bool valid = row < M;
    const int rr = valid ? row : M - 1;
    const int i = rr / p, jp = rr - i * p;
    const uint16_t* qr = P.q + ((size_t)i * P.h + (size_t)gam * p + jp) * D;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) qop[ks] = load16(qr + 16 * ks + 8 * h);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
      for (int w = 0; w < 4; ++w) qop[ks][w] = valid ? qop[ks][w] ^ P.q_sign : 0u;
  }
  // Code caches: load q = tid + 64 NW u of a stage reads 16 bytes of codes
  // (E elements, chunk c16 of row `row` of K, then of V) and writes them,
  // widened, as E / 8 bf16 slots of that row in LDS.
  constexpr int E = 128 / KV::BITS;        // elements per 16-byte load
  constexpr int CPR = CRB / 16;            // loads per row
  constexpr int SLOADS = 2 * SK * CPR;     // loads per stage
  constexpr int SPT = kDirect ? 1 : (SLOADS + 64 * NW - 1) / (64 * NW);  // per thread
  static_assert(kDirect || SLOADS % (64 * NW) == 0, "whole loads per thread");
  u32x4 sreg[SPT];
  auto stage_get = [&](int key0) {
    const int rows = nkeys - key0;
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(kchunk + (size_t)key0 * CRB, rows, CRB);
    const __amdgpu_buffer_rsrc_t rv = rows_rsrc(vchunk + (size_t)key0 * CRB, rows, CRB);
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int q = (int)threadIdx.x + 64 * NW * u;
      const bool is_v = q >= SK * CPR;  // wave-uniform: whole waves per half
      const int qq = is_v ? q - SK * CPR : q;
      sreg[u] = Raw<16>::load(is_v ? rv : rk, boff((uint32_t)qq * 16));
    }
  };
  auto stage_put = [&](int buf) {
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int q = (int)threadIdx.x + 64 * NW * u;
      const bool is_v = q >= SK * CPR;
      const int qq = is_v ? q - SK * CPR : q;
      const int row = qq / CPR, c16 = qq % CPR;
      unsigned char* dst = lds + buf * STAGE + (is_v ? KAREA + row * VROW : row * KROW) + c16 * E * 2;
      const u32x4& w = sreg[u];
      if constexpr (KV::BITS == 8) {
        *(lds_u32x4*)dst = Widen8<KV>::run(u32x2{w[0], w[1]});
        *(lds_u32x4*)(dst + 16) = Widen8<KV>::run(u32x2{w[2], w[3]});
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) *(lds_u32x4*)(dst + 16 * k) = Widen8<KV>::run(w[k]);
      }
    }
  };
  const int nstages = (nkeys + SK - 1) / SK;
  if constexpr (kDirect) {
#pragma unroll
    for (int t = 0; t < NB - 1; ++t)
      if (t < nstages) fetch(t * SK, t);
  } else {
    stage_get(0);
    stage_put(0);
    if (nstages > 1) stage_get(SK);
  }

  // Per-lane LDS read bases (from a stage buffer's start): key operand of row
  // j, half h; value chunk of key 4(q/2) + i'/4, dims 16(q%2) + 4(i'%4).
  const int q4 = lane >> 4, ip = lane & 15;
  const int kbase = j * KROW + h * 16;
  const int vbase = KAREA + (4 * (q4 >> 1) + (ip >> 2)) * VROW + (16 * (q4 & 1) + 4 * (ip & 3)) * 2;

  f32x16 acc[DB];
#pragma unroll
  for (int t = 0; t < DB; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
  float mref = kNegInf, lsum = 0.f;
  const bool active = row0 < M;  // wave-uniform

  for (int st = 0; st < nstages; ++st) {
    const int buf = st % NB;
    if constexpr (kDirect) {
      // After this wave's wait, the barrier hands every wave's part of stage
      // st to all waves and frees buffer (st - 1) % NB, which all have read.
      wait_stage(st + 1 >= nstages);
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      if (st + NB - 1 < nstages) fetch((st + NB - 1) * SK, (st + NB - 1) % NB);
    } else {
      // The barrier hands stage st (written from registers) to all waves and
      // frees the other buffer: stage st + 1 goes there from the registers
      // loaded a stage ago, and stage st + 2 is loaded into them.
      __syncthreads();
      if (st + 1 < nstages) {
        stage_put(buf ^ 1);
        if (st + 2 < nstages) stage_get((st + 2) * SK);
      }
    }
    if (!active) continue;
    const unsigned char* kb = lds + buf * STAGE + kbase;
    const uint32_t vaddr = (uint32_t)(uintptr_t)(lds_void*)(lds + buf * STAGE + vbase);
    const int rem = nkeys - st * SK;  // valid keys from the stage's first
    // The key operands of block 0 of the stage; each later block's are read
    // during the previous block's value products.
    const uint32_t kaddr = (uint32_t)(uintptr_t)(lds_void*)(kb);
    u32x4 kw[KSTEPS];
    read_k_block(kaddr, kw);
    lds_wait_k(kw);
#pragma unroll
    for (int b = 0; b < SK / 32; ++b) {
      // S^T block: keys 32b .. 32b+31 of the stage
      f32x16 sacc;
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) sacc = mfma32(kw[ks], qop[ks], sacc);
      // this block's V^T operands, read while the weights are formed (after
      // the key operand reads, whose waits would otherwise cover them too)
      __builtin_amdgcn_sched_barrier(0);
      u32x2 vw[16];
      read_vt_block<VROW>(vaddr + 32 * b * VROW, vw);
      float x[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) x[v] = sacc[v];
      if (rem < 32 * (b + 1)) {
        const int nv = __builtin_amdgcn_readfirstlane(rem) - 32 * b;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (8 * (v / 4) + 4 * h + (v & 3) >= nv) x[v] = kNegInf;
      }
      // Weights against the current reference first: while their sum stays
      // within 2^kRescaleSlack no weight exceeds it, and the reference keeps
      // its value (a raise needs a weight above 2^kRescaleSlack). Otherwise,
      // and on the first block, the row's maximum decides the raise and the
      // weights are formed again.
      float pr[16];
      float ps;
      {
        const float nbase = mref == kNegInf ? 0.f : -mref;
#pragma unroll
        for (int v = 0; v < 16; ++v) pr[v] = exp2_fast(__builtin_fmaf(x[v], sl2, nbase));
        ps = pr[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) ps += pr[v];
      }
      if (__any(!(ps <= kSumBound) || mref == kNegInf)) {
        float lmax = x[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) lmax = fmaxf(lmax, x[v]);
        const float tmax = xor32_max(lmax) * sl2;  // the row's maximum over the block
        const bool raise = tmax > mref + kRescaleSlack;
        if (__any(raise)) {
          const float alpha = raise ? exp2_fast(mref - tmax) : 1.f;
          lsum *= alpha;
#pragma unroll
          for (int t = 0; t < DB; ++t) acc[t] *= alpha;
          mref = raise ? tmax : mref;
          const float nbase = mref == kNegInf ? 0.f : -mref;
#pragma unroll
          for (int v = 0; v < 16; ++v) pr[v] = exp2_fast(__builtin_fmaf(x[v], sl2, nbase));
          ps = pr[0];
#pragma unroll
          for (int v = 1; v < 16; ++v) ps += pr[v];
        }
      }
      lsum += ps;
      u32x4 pb[2];
#pragma unroll
      for (int ss = 0; ss < 2; ++ss)
#pragma unroll
        for (int w = 0; w < 4; ++w) pb[ss][w] = pack_bf16(pr[8 * ss + 2 * w], pr[8 * ss + 2 * w + 1]);
      // O^T += V^T P^T, dims 32t .. 32t+31, keys of k-step ss
      lds_wait_tr(vw);
      if (b + 1 < SK / 32) read_k_block(kaddr + 32 * (b + 1) * KROW, kw);
#pragma unroll
      for (int ss = 0; ss < 2; ++ss)
#pragma unroll
        for (int t = 0; t < DB; ++t) {
          const u32x2 lo = vw[8 * ss + 2 * t], hi = vw[8 * ss + 2 * t + 1];
          acc[t] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb[ss], acc[t]);
        }
      if (b + 1 < SK / 32) lds_wait_k(kw);
    }
  }

  if (!active) return;
  const float ltot = xor32_sum(lsum);
  const int row = row0 + j;
  if (row < M) {
    const size_t prow = ((size_t)gam * P.S_c + s) * P.M + row;
    float* dst = P.ctx_acc + prow * D;
#pragma unroll
    for (int t = 0; t < DB; ++t)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *reinterpret_cast<f32x4*>(dst + 32 * t + 8 * g4 + 4 * h) =
            f32x4{acc[t][4 * g4], acc[t][4 * g4 + 1], acc[t][4 * g4 + 2], acc[t][4 * g4 + 3]};
    if (h == 0) P.ctx_ml[prow] = float2{mref, ltot};
  }
}

template <int NW, int NB, int SK, typename KV>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void
ctx_wide_kernel(PartialsParams P) {
  ctx_wide_body<NW, NB, SK, KV>(P);
}



// Grid: n_ctx_small_blocks work-groups of the few-row context path, then
// n_dec_blocks decode work-groups (the many-row context path has a kernel of
// its own).
template <int D, typename KV, int CTX, int NTD>
__device__ __forceinline__ void partials_body(const PartialsParams& P) {
  constexpr bool kSmall = CTX != kCtxNone;
  constexpr int NTC = kSmall ? CTX : 1;
  constexpr int NTQ = NTC > NTD ? NTC : NTD;
  constexpr int QSLOTS = kWaves * NTQ * (D / 32) * 64;  // u32x4 slots for Q^T operands
  constexpr int KSLOTS = kWaves * kTileKeys * D / 8;      // one staged K tile per wave
  constexpr int MERGE = kSmall ? (MergeLds<D, NTC>::bytes + 15) / 16 : 0;  // overlays the K tiles
  constexpr int LDS = QSLOTS + cmax(KSLOTS, MERGE);
  __shared__ __attribute__((aligned(16))) u32x4 lds[LDS];
  const int bid = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = wave_id();
  u32x4* qw = lds + wave * NTQ * (D / 32) * 64;
  u32x4* kl = lds + QSLOTS + wave * (kTileKeys * D / 8);
  const int blk = bid;
  if (blk < P.n_ctx_small_blocks) {
    if constexpr (kSmall)
      ctx_small_block<D, NTC, KV>(P, blk, wave, lane, qw, kl,
                                  reinterpret_cast<float*>(lds + QSLOTS));
  } else if (blk - P.n_ctx_small_blocks < P.n_dec_blocks) {
    decode_block<D, NTD, KV>(P, blk - P.n_ctx_small_blocks, wave, lane, qw, kl);
  }
}

// Variants whose waves hold at most two query tiles fit two waves
// per SIMD (<= 256 registers) and are compiled for that occupancy; the others
// keep the compiler's choice.
template <int D, typename KV, int CTX, int NTD>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void
partials_kernel_2w(PartialsParams P) {
  partials_body<D, KV, CTX, NTD>(P);
}
template <int D, typename KV, int CTX, int NTD>
__global__ __launch_bounds__(kThreads) void partials_kernel(PartialsParams P) {
  partials_body<D, KV, CTX, NTD>(P);
}
template <int D, int CTX, int NTD>
constexpr bool fits_two_waves() {
  return CTX != kCtxSmall4 && NTD <= 2;
}

// Combine (the joint softmax of Eq. 3-4): one wave per output row (i, j)
// merges the row's context partials (group j/p, every split) and decode
// partials (sample i, group j/p, every chunk; empty ones weigh 0) into
// out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k, M = max_k m_k.
// Lane k first fetches the statistics of partial k (all in parallel), so the
// weights need one wave reduction; the value rows are then summed in a fixed
// order with their loads issued ahead in batches. The group's value scale
// multiplies the result (every partial of the row shares it); the first row
// of each group checks that the group's scales are positive normal floats.
template <int D, int BATCH>
__global__ __launch_bounds__(256) void combine_kernel(CombineParams C) {
  constexpr int PER = D / 64;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int row = blockIdx.x * 4 + wave;
  if (row >= C.b * C.h) return;
  const int i = row / C.h, j = row - i * C.h;
  const int gam = j / C.p, jp = j - gam * C.p;
  if (j == 0 && lane == 0 && C.lens) {
    const int raw = C.lens[i];
    if (raw < 0 || raw > C.m_d_max) atomicOr(C.status, kStatusLens);
  }
  const float vs = C.v_scale ? C.v_scale[gam] : 1.f;
  if (i == 0 && jp == 0 && lane == 0) {
    const float ks = C.k_scale ? C.k_scale[gam] : 1.f;
    // false for NaN as well
    const bool ok = ks >= __FLT_MIN__ && ks <= __FLT_MAX__ && vs >= __FLT_MIN__ && vs <= __FLT_MAX__;
    if (!ok) atomicOr(C.status, kStatusScale);
  }
  const int np = C.S_c + C.S_d;  // every decode wave wrote a partial (maybe empty)
  const size_t cbase = (size_t)gam * C.S_c * C.M + (size_t)i * C.p + jp;  // + k*M
  const size_t dbase = ((size_t)(i * C.g + gam) * C.S_d) * C.p + jp;      // + k*p
  auto idx = [&](int k) -> size_t {
    return k < C.S_c ? cbase + (size_t)k * C.M : dbase + (size_t)(k - C.S_c) * C.p;
  };
  auto accp = [&](int k) -> const float* {
    return (k < C.S_c ? C.ctx_acc : C.dec_acc) + idx(k) * D + lane * PER;
  };
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  float L = 0.f;
  float mx = kNegInf;
  for (int k0 = 0; k0 < np; k0 += 64) {  // running max over chunks of 64 partials
    const int kn = min(64, np - k0);
    // Issue the first batch of value rows together with the statistics, so
    // a chunk of up to BATCH partials costs one memory round trip; only the
    // rows the chunk has are loaded (kn is wave-uniform).
    float v[BATCH][PER];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      if (u < kn) {
        const float* a = accp(k0 + u);
#pragma unroll
        for (int e = 0; e < PER; ++e) v[u][e] = a[e];
      }
    }
    const int k = k0 + lane;
    const float2 ml = k < np ? (k < C.S_c ? C.ctx_ml[idx(k)] : C.dec_ml[idx(k)])
                             : float2{kNegInf, 0.f};
    float cm = ml.x;
    cm = wave_max(cm);
    const float mnew = fmaxf(mx, cm);
    const float base = mnew == kNegInf ? 0.f : mnew;
    const float rescale = exp2_fast(mx - base);  // 0 on the first chunk
    L *= rescale;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] *= rescale;
    mx = mnew;
    const float w = exp2_fast(ml.x - base);      // 0 for padding lanes
    float lw = w * ml.y;
    lw = wave_sum(lw);
    L += lw;
    for (int kb = 0; kb < kn; kb += BATCH) {
      if (kb > 0) {
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
          if (kb + u < kn) {
            const float* a = accp(k0 + kb + u);
#pragma unroll
            for (int e = 0; e < PER; ++e) v[u][e] = a[e];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const float wu = __shfl(w, min(kb + u, 63));
        if (kb + u < kn) {
#pragma unroll
          for (int e = 0; e < PER; ++e) acc[e] += wu * v[u][e];
        }
      }
    }
  }
  float* o = C.out + (size_t)row * D + lane * PER;
  const float inv = vs / L;
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = acc[e] * inv;
}

// One launch; with events, through hipExtLaunchKernel so that they carry the
// kernel's own start and end.
template <typename Prm>
hipError_t launch(void (*kernel)(Prm), int grid, int block, hipStream_t stream,
                  const LaunchEvents& ev, const Prm& p) {
  if (ev.start || ev.stop)
    hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(block), 0, stream, ev.start, ev.stop, 0, p);
  else
    kernel<<<grid, block, 0, stream>>>(p);
  return hipGetLastError();
}

template <int D, typename KV, int CTX>
hipError_t launch_partials_ctx(const PartialsParams& P, int dec_tiles, hipStream_t stream,
                               const LaunchEvents& ev) {
  const int grid = P.n_ctx_small_blocks + P.n_dec_blocks;
  if (grid == 0) return hipSuccess;
  switch (dec_tiles) {
    case 1:
      if constexpr (fits_two_waves<D, CTX, 1>())
        return launch(partials_kernel_2w<D, KV, CTX, 1>, grid, kThreads, stream, ev, P);
      else
        return launch(partials_kernel<D, KV, CTX, 1>, grid, kThreads, stream, ev, P);
    case 2:
      if constexpr (fits_two_waves<D, CTX, 2>())
        return launch(partials_kernel_2w<D, KV, CTX, 2>, grid, kThreads, stream, ev, P);
      else
        return launch(partials_kernel<D, KV, CTX, 2>, grid, kThreads, stream, ev, P);
    case 4: return launch(partials_kernel<D, KV, CTX, 4>, grid, kThreads, stream, ev, P);
    default: return hipErrorInvalidValue;
  }
}

template <int D, typename KV>
hipError_t launch_partials_dk(const PartialsParams& P, int ctx_mode, int dec_tiles,
                              hipStream_t stream, const LaunchEvents& ev) {
  switch (ctx_mode) {
    case kCtxNone: return launch_partials_ctx<D, KV, kCtxNone>(P, dec_tiles, stream, ev);
    case kCtxSmall1: return launch_partials_ctx<D, KV, kCtxSmall1>(P, dec_tiles, stream, ev);
    case kCtxSmall2: return launch_partials_ctx<D, KV, kCtxSmall2>(P, dec_tiles, stream, ev);
    case kCtxSmall4: return launch_partials_ctx<D, KV, kCtxSmall4>(P, dec_tiles, stream, ev);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t launch_partials_d(const PartialsParams& P, int kv, int ctx_mode, int dec_tiles,
                             hipStream_t stream, const LaunchEvents& ev) {
  switch (kv) {
    case kKvBf16: return launch_partials_dk<D, KvBf16>(P, ctx_mode, dec_tiles, stream, ev);
    case kKvFp8: return launch_partials_dk<D, KvFp8>(P, ctx_mode, dec_tiles, stream, ev);
    case kKvInt8: return launch_partials_dk<D, KvInt8>(P, ctx_mode, dec_tiles, stream, ev);
    case kKvInt4: return launch_partials_dk<D, KvInt4>(P, ctx_mode, dec_tiles, stream, ev);
    default: return hipErrorInvalidValue;
  }
}

template <int D, typename KV>
hipError_t launch_standard_dk(const PartialsParams& P, int tiles, hipStream_t stream,
                              const LaunchEvents& ev) {
  const int grid = P.b * P.g;
  switch (tiles) {
    case 1: return launch(standard_kernel<D, 1, KV>, grid, kThreads, stream, ev, P);
    case 2: return launch(standard_kernel<D, 2, KV>, grid, kThreads, stream, ev, P);
    case 4: return launch(standard_kernel<D, 4, KV>, grid, kThreads, stream, ev, P);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t launch_standard_d(const PartialsParams& P, int kv, int tiles, hipStream_t stream,
                             const LaunchEvents& ev) {
  switch (kv) {
    case kKvBf16: return launch_standard_dk<D, KvBf16>(P, tiles, stream, ev);
    case kKvFp8: return launch_standard_dk<D, KvFp8>(P, tiles, stream, ev);
    case kKvInt8: return launch_standard_dk<D, KvInt8>(P, tiles, stream, ev);
    case kKvInt4: return launch_standard_dk<D, KvInt4>(P, tiles, stream, ev);
    default: return hipErrorInvalidValue;
  }
}

template <typename KV>
hipError_t launch_ctx_wide_kv(const PartialsParams& P, hipStream_t stream,
                              const LaunchEvents& ev) {
  constexpr bool kDirect = KV::BITS == 16;
  // eight waves: 128-key stages, two in LDS (fewer barriers than 64-key
  // stages, measured 3-5% faster); chunks of a multiple of 64 keys (three
  // 64-key stages in LDS for bf16, two for code caches, which stage a
  // third in registers)
  if (P.ctx_wide == 8) {
    if (P.ctx_keys % 128 == 0)
      return launch(ctx_wide_kernel<8, 2, 128, KV>, P.n_ctx_blocks, 512, stream, ev, P);
    return launch(ctx_wide_kernel<8, kDirect ? 3 : 2, 64, KV>, P.n_ctx_blocks, 512, stream, ev, P);
  }
  if (P.ctx_wide == 4) return launch(ctx_wide_kernel<4, 2, 64, KV>, P.n_ctx_blocks, 256, stream, ev, P);
  return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_ctx_large_d(const PartialsParams& P, int kv, hipStream_t stream,
                              const LaunchEvents& ev) {
  const int grid = P.n_ctx_blocks;
  switch (kv) {
    case kKvBf16: return launch(ctx_large_kernel<D, KvBf16>, grid, kLargeThreads, stream, ev, P);
    case kKvFp8: return launch(ctx_large_kernel<D, KvFp8>, grid, kLargeThreads, stream, ev, P);
    case kKvInt8: return launch(ctx_large_kernel<D, KvInt8>, grid, kLargeThreads, stream, ev, P);
    case kKvInt4: return launch(ctx_large_kernel<D, KvInt4>, grid, kLargeThreads, stream, ev, P);
    default: return hipErrorInvalidValue;
  }
}

// Decode-cache append (the decode cache holds the keys and values of the
// previous decoding steps, Section 3.1): work-group i copies sample i's n new
// rows of every group to rows len_i .. len_i + n - 1 of its decode cache and
// then advances len_i by n. One work-group per sample, so every thread reads
// len_i before thread 0 rewrites it. Rows past the capacity are dropped; a
// length outside [0, m_d_max] is clamped; both raise the status flag. RB:
// bytes per row (elements of the cache type, copied as they are).
template <int RB>
__global__ __launch_bounds__(256) void append_kernel(AppendParams A) {
  constexpr int CH = RB / 16;  // 16-byte chunks per row
  const int i = blockIdx.x;
  const int raw = A.lens[i];
  const int len = raw < 0 ? 0 : (raw > A.m_d_max ? A.m_d_max : raw);
  const int room = min(A.n, A.m_d_max - len);  // new rows that fit
  const int total = A.g * room * CH;
  for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
    const int c = idx % CH;
    const int r = (idx / CH) % room;
    const int gam = idx / CH / room;
    const size_t unit = (size_t)i * A.g + gam;
    const size_t src = (unit * A.n + r) * RB + c * 16;
    const size_t dst = (unit * A.m_d_max + len + r) * RB + c * 16;
    *reinterpret_cast<u32x4*>(A.Kd + dst) = *reinterpret_cast<const u32x4*>(A.k_new + src);
    *reinterpret_cast<u32x4*>(A.Vd + dst) = *reinterpret_cast<const u32x4*>(A.v_new + src);
  }
  __syncthreads();  // every thread has read len_i
  if (threadIdx.x == 0) {
    if (raw != len || room < A.n) atomicOr(A.status, kStatusLens);
    A.lens[i] = len + room;
  }
}

}  // namespace

hipError_t launch_append(const AppendParams& A, int d, int kv, hipStream_t stream,
                         const LaunchEvents& ev) {
  switch (kv_row_bytes(d, kv)) {
    case 256: return launch(append_kernel<256>, A.b, 256, stream, ev, A);
    case 128: return launch(append_kernel<128>, A.b, 256, stream, ev, A);
    case 64: return launch(append_kernel<64>, A.b, 256, stream, ev, A);
    case 32: return launch(append_kernel<32>, A.b, 256, stream, ev, A);
    default: return hipErrorInvalidValue;
  }
}
// Scratch of the allocation-free entry point (partials and the status word
// of one call). In host code `scratch` names a host-side stand-in, not the
// device memory: its device address comes from hipGetSymbolAddress, per
// device, and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_address(int device, void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // looked up with its device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *ptr = addr[device];
  return hipSuccess;
}

hipError_t launch_ctx_large(const PartialsParams& P, int d, int kv, hipStream_t stream,
                            const LaunchEvents& ev) {
  if (P.n_ctx_blocks == 0) return hipSuccess;
  if (P.ctx_wide) {
    if (d != 128) return hipErrorInvalidValue;
    switch (kv) {
      case kKvBf16: return launch_ctx_wide_kv<KvBf16>(P, stream, ev);
      case kKvFp8: return launch_ctx_wide_kv<KvFp8>(P, stream, ev);
      case kKvInt8: return launch_ctx_wide_kv<KvInt8>(P, stream, ev);
      case kKvInt4: return launch_ctx_wide_kv<KvInt4>(P, stream, ev);
      default: return hipErrorInvalidValue;
    }
  }
  if (d == 128) return launch_ctx_large_d<128>(P, kv, stream, ev);
  if (d == 64) return launch_ctx_large_d<64>(P, kv, stream, ev);
  return hipErrorInvalidValue;
}
hipError_t launch_standard(const PartialsParams& P, int d, int kv, int tiles,
                           hipStream_t stream, const LaunchEvents& ev) {
  if (P.b * P.g == 0) return hipSuccess;
  if (d == 128) return launch_standard_d<128>(P, kv, tiles, stream, ev);
  if (d == 64) return launch_standard_d<64>(P, kv, tiles, stream, ev);
  return hipErrorInvalidValue;
}
hipError_t launch_partials(const PartialsParams& P, int d, int kv, int ctx_mode, int dec_tiles,
                           hipStream_t stream, const LaunchEvents& ev) {
  if (d == 128) return launch_partials_d<128>(P, kv, ctx_mode, dec_tiles, stream, ev);
  if (d == 64) return launch_partials_d<64>(P, kv, ctx_mode, dec_tiles, stream, ev);
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const CombineParams& C, int d, hipStream_t stream,
                          const LaunchEvents& ev) {
  const int rows = C.b * C.h;
  const int grid = (rows + 3) / 4;
  // One batch of value rows holds every partial of a row where it has at
  // most 32 (one memory round trip), in the smallest of 8, 16, 32 rows.
  const int np = C.S_c + C.S_d;
  if (d == 128)
    return np <= 8 ? launch(combine_kernel<128, 8>, grid, 256, stream, ev, C)
         : np <= 16 ? launch(combine_kernel<128, 16>, grid, 256, stream, ev, C)
                    : launch(combine_kernel<128, 32>, grid, 256, stream, ev, C);
  if (d == 64)
    return np <= 8 ? launch(combine_kernel<64, 8>, grid, 256, stream, ev, C)
         : np <= 16 ? launch(combine_kernel<64, 16>, grid, 256, stream, ev, C)
                    : launch(combine_kernel<64, 32>, grid, 256, stream, ev, C);
  return hipErrorInvalidValue;
}

}  // namespace bifattn

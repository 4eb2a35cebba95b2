// HIP kernels of the compose-and-attend path for gfx950 (CDNA4).
//
//   compose_kernel   blender B (Section 2.2, Eq. 3; Section 3.2; Appendix C):
//                    gather kept rows -> decode (int8 * scale) -> turn keys by
//                    their segment's delta -> write pages (V transposed in-page)
//   attn_kernel      attention of the query tokens over [KV_total, x_q]
//                    (Eq. 4): suffix RoPE on load, MFMA S^T = K Q^T, online
//                    softmax in base 2, MFMA O^T = V^T P^T; keys come from the
//                    pages, or straight from the pool (gather/decode/turn fused)
//   merge_kernel     log-sum-exp combine of key splits, a thread per output
//                    element; merge_split_kernel: one row per workgroup with
//                    the splits spread over its lanes (many splits, few rows)
//
// MFMA use.  One wavefront owns 32 query rows.  Scores are computed transposed
// (keys x queries) so that in the 32x32 accumulator layout every lane holds one
// query's scores: the row max needs a single exchange between the two 32-lane
// halves, and the probabilities feed the P*V product from the lane that holds
// them.  The contraction index of P*V (the key) is permuted to follow that
// accumulator layout; V^T is read from LDS with the same permutation.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>

#include "plan.hpp"

namespace c2kv {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int KT = kKeyTile;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLazyLog2 = 8.f;  // reference-maximum slack of the bf16 online softmax
constexpr float kLn2 = 0.693147180559945309f;
// fourth descriptor word of a raw (unformatted, unswizzled) buffer on gfx9-family
// parts; reads past num_records return zero
constexpr int kBufferFlags = 0x00020000;
// row blocks (of at most 128 rows) with more splits than this are merged one
// row per workgroup
constexpr int kSplitMergeMin = 16;

// SRC_PAGED_SIF: pages, with the Structured Information Flow mask over the
// suffix instead of the causal one (its own kernels, so that the causal ones
// carry none of the SIF mask's registers)
enum Src { SRC_PAGED = 0, SRC_POOL = 1, SRC_POOL_I8 = 2, SRC_PAGED_SIF = 3 };

// ----------------------------------------------------------------------------
// element helpers
// ----------------------------------------------------------------------------

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(__bf16 x) { return static_cast<float>(x); }

template <typename T> __device__ inline T from_f(float x);
template <> __device__ inline float from_f<float>(float x) { return x; }
template <> __device__ inline __bf16 from_f<__bf16>(float x) { return static_cast<__bf16>(x); }

// 8 consecutive elements -> float
__device__ inline void load8(const float* p, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ inline void load8(const __bf16* p, float (&x)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ inline void load8(const int8_t* p, float (&x)[8]) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[i] = static_cast<float>(static_cast<int8_t>((u.x >> (8 * i)) & 0xff));
    x[4 + i] = static_cast<float>(static_cast<int8_t>((u.y >> (8 * i)) & 0xff));
  }
}

// 8 floats -> 8 consecutive T (16-byte aligned destination for bf16)
__device__ inline void store8(float* p, const float (&x)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
// (a, b) -> bf16 pair, a in the low half: one paired round-to-nearest-even
// conversion (two scalar conversions would each need a shift or merge after)
__device__ inline uint32_t pack_bf16(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ inline void store8(__bf16* p, const float (&x)[8]) {
  uint4 u;
  u.x = pack_bf16(x[0], x[1]);
  u.y = pack_bf16(x[2], x[3]);
  u.z = pack_bf16(x[4], x[5]);
  u.w = pack_bf16(x[6], x[7]);
  *reinterpret_cast<uint4*>(p) = u;
}
template <typename T>
__device__ inline void store8_zero(T* p) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(p + 4) = make_float4(0.f, 0.f, 0.f, 0.f);
  } else {
    *reinterpret_cast<uint4*>(p) = make_uint4(0u, 0u, 0u, 0u);
  }
}

// cos/sin of 8 consecutive frequencies (float2 pairs)
__device__ inline void load_cs8(const float2* cs, float (&c)[8], float (&s)[8]) {
  const float4* p = reinterpret_cast<const float4*>(cs);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float4 v = p[i];
    c[2 * i] = v.x; s[2 * i] = v.y; c[2 * i + 1] = v.z; s[2 * i + 1] = v.w;
  }
}

// Half-split RoPE turn of the pair (x_i, x_{i+D/2}) by the angle whose cos/sin
// are given (x <- x c - y s, y <- x s + y c).  The fused multiply-adds are
// written out so that every kernel rounds a turned key the same way.
__device__ inline void rotate_pair(float& x, float& y, float c, float s) {
  const float a = x, b = y;
  x = __builtin_fmaf(a, c, -(b * s));
  y = __builtin_fmaf(a, s, b * c);
}
__device__ inline void rotate8(float (&x)[8], float (&y)[8], const float (&c)[8],
                               const float (&s)[8]) {
#pragma unroll
  for (int e = 0; e < 8; ++e) rotate_pair(x[e], y[e], c[e], s[e]);
}

// ----------------------------------------------------------------------------
// MFMA traits: bf16 32x32x16 (8 k per lane) and f32 32x32x2 (1 k per lane)
// ----------------------------------------------------------------------------

template <typename T> struct Mma;
template <> struct Mma<float> {
  static constexpr int KPL = 1;
  using Op = float;
  __device__ static inline f32x16 run(Op a, Op b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma<__bf16> {
  static constexpr int KPL = 8;
  using Op = bf16x8;
  __device__ static inline f32x16 run(Op a, Op b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

// maximum of x over lanes l and l ^ 32, a VALU lane swap: the swap's first
// result holds the lower half's values in every lane, the second the upper's
__device__ inline float half_pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// sum of x over lanes l and l ^ 32, the same value (same operand order) in both
__device__ inline float half_pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ----------------------------------------------------------------------------
// raw 32-bit words of 8 consecutive elements (2 * sizeof(S) words)
// ----------------------------------------------------------------------------

template <typename S>
__device__ inline void raw_load8(uint32_t* w, const S* p) {
  if constexpr (sizeof(S) == 4) {
    const uint4 u0 = *reinterpret_cast<const uint4*>(p);
    const uint4 u1 = *reinterpret_cast<const uint4*>(p + 4);
    w[0] = u0.x; w[1] = u0.y; w[2] = u0.z; w[3] = u0.w;
    w[4] = u1.x; w[5] = u1.y; w[6] = u1.z; w[7] = u1.w;
  } else if constexpr (sizeof(S) == 2) {
    const uint4 u0 = *reinterpret_cast<const uint4*>(p);
    w[0] = u0.x; w[1] = u0.y; w[2] = u0.z; w[3] = u0.w;
  } else {
    const uint2 u0 = *reinterpret_cast<const uint2*>(p);
    w[0] = u0.x; w[1] = u0.y;
  }
}
template <typename S>
__device__ inline void raw_zero8(uint32_t* w) {
#pragma unroll
  for (int i = 0; i < 2 * int(sizeof(S)); ++i) w[i] = 0u;
}
template <typename S>
__device__ inline void raw_to_f8(const uint32_t* w, float (&x)[8]) {
  if constexpr (sizeof(S) == 4) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __uint_as_float(w[i]);
  } else if constexpr (sizeof(S) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      x[i] = static_cast<float>(static_cast<int8_t>((w[i >> 2] >> (8 * (i & 3))) & 0xffu));
  }
}

// zero the elements [n_keep, 16 / sizeof(T)) of a 16-byte vector (a mask per
// word from selects, no branches: n_keep differs between lanes)
template <typename T>
__device__ inline uint4 keep_first(uint4 v, int n_keep) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
  constexpr int EPW = 4 / sizeof(T);              // elements per word
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int k = n_keep - EPW * i;               // elements of word i to keep
    uint32_t m = k >= EPW ? 0xffffffffu : 0u;
    if constexpr (EPW == 2) m = k == 1 ? 0x0000ffffu : m;
    w[i] &= m;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ----------------------------------------------------------------------------
// parameters
// ----------------------------------------------------------------------------

struct AttnParams {
  int Hq, Hkv, G, S, PS, max_pages, RB, n_seg, merge_in_kernel;
  int sif_n, sif_block, sif_sink;  // SIF mask over the suffix when sif_n > 0
  int tpp;                      // key tiles per page (PS / KT)
  unsigned tpp_magic;           // floor(2^32 / tpp) + 1 (tpp > 1)
  float qscale;                 // softmax scale * log2(e)
  const int* req_slot0;
  const int2* slot_info;        // (pool row, segment) per composed slot
  const float2* seg_cs;         // [n_seg][D/2] cos/sin(delta * theta_i)
  const float2* suf_cs;         // [B][S][D/2]  cos/sin((span_end + t) * theta_i)
  const int* block_table;
  const WorkItem* items;
  const MergeGroup* merges;
  int* counters;                // [n_merge], zero between launches
  const void* k;                // pages or pool
  const void* v;
  const float* k_scale;
  const float* v_scale;
  const void* q;
  const void* k_suf;
  const void* v_suf;
  void* out;
  float* lse;
  void* part_o;                 // [n_partials][RB][D], activation dtype
  float* part_lse;
};

struct ComposeParams {
  int Hkv, PS;
  const int2* slot_info;
  const int* slot_pos;
  const float2* seg_cs;
  const int4* tiles;           // [n] (first slot, keys in the tile, page, offset in it)
  const void* k;               // pool
  const void* v;
  const float* k_scale;
  const float* v_scale;
  void* k_pages;
  void* v_pages;
  int64_t* out_src_row;        // optional
  int32_t* out_pos;            // optional
};

struct MergeParams {
  int Hq, G, S, RB;
  const MergeGroup* groups;
  const void* part_o;
  const float* part_lse;
  void* out;
  float* lse;
};

template <typename T, int D>
struct Lds {
  // keys: rows of D elements padded by 16 bytes (16-byte reads, 4-bank row shift).
  // Transposed values, bf16: rows of KT keys padded by 16 bytes, with the keys of
  // each group of 16 stored in the order 0-3, 8-11, 4-7, 12-15, so that the 8 keys
  // one lane feeds to a P*V product (4h..4h+3 and 8+4h..8+4h+3 of a group, h the
  // lane's half) are one 16-byte read; 16 consecutive rows of such reads fall on
  // distinct banks.  fp32: rows padded by 8 bytes, natural key order.
  static constexpr int LDK = D + 16 / int(sizeof(T));
  static constexpr int LDV = KT + (sizeof(T) == 2 ? 16 : 8) / int(sizeof(T));
  static constexpr int TILE = KT * LDK + D * LDV;   // elements of one stage
  // column of key k in a transposed value row (swaps bits 2 and 3 of k for bf16)
  __device__ static constexpr int vcol(int k) {
    return sizeof(T) == 2 ? (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1) : k;
  }
};

constexpr int imax(int a, int b) { return a > b ? a : b; }

// Per-thread work of one key tile for an NT-thread workgroup.
template <typename T, typename PoolT, int D, int NT, bool PAGED>
struct Shape {
  static constexpr int KU_TOT = KT * (D / 16);     // key units: (chunk, chunk + D/2) pairs
  static constexpr int VU_TOT = (KT / 2) * (D / 8);// value units: 8-element chunk of 2 keys
  static constexpr int NKU = (KU_TOT + NT - 1) / NT;
  static constexpr int NVU = (VU_TOT + NT - 1) / NT;
  // every thread's units all inside the tile: no per-unit guard (a guarded
  // load leaves the compiler's wait counts conservative after it)
  static constexpr bool KU_ALL = KU_TOT % NT == 0;
  static constexpr bool VU_ALL = VU_TOT % NT == 0;
  static constexpr int EPV = 16 / sizeof(T);       // elements per 16-byte vector
  static constexpr int PK_TOT = KT * D / EPV;      // page vectors, keys
  static constexpr int PV_TOT = D * KT / EPV;      // page vectors, transposed values
  static constexpr int NPK = (PK_TOT + NT - 1) / NT;
  static constexpr int NPV = (PV_TOT + NT - 1) / NT;
  static constexpr int WP = 2 * int(sizeof(PoolT));    // words per 8 pool elements
  static constexpr int WA = 2 * int(sizeof(T));        // words per 8 act elements
  static constexpr int RKW = imax(NKU * 2 * WA, PAGED ? NPK * 4 : NKU * 2 * WP);
  static constexpr int RVW = imax(NVU * 2 * WA, PAGED ? NPV * 4 : NVU * 2 * WP);
};

// The suffix keys a query row sees, as ranges fixed per row.  Causal: keys
// [0, t].  Structured Information Flow over the sequence [n originals | C^2
// tokens]: an original t sees originals [0, t]; C^2 token j = t - n sees C^2
// tokens [n, t], the sink [0, sif_sink) and the originals of its block
// [j*block, min((j+1)*block, n)).
struct RowKeys {
  int lo, hi;          // [lo, hi], inclusive
  int sink;            // [0, sink)
  int blo, bhi;        // [blo, bhi)
  __device__ RowKeys(int t, const AttnParams& a) {
    lo = 0; hi = t; sink = 0; blo = 0; bhi = 0;
    if (a.sif_n > 0 && t >= a.sif_n) {
      const int j = t - a.sif_n;
      lo = a.sif_n;
      sink = a.sif_sink;
      blo = j * a.sif_block;
      bhi = min((j + 1) * a.sif_block, a.sif_n);
    }
  }
  // each range test is one unsigned compare of u - start against the length
  __device__ bool sees(int u) const {
    return unsigned(u - lo) <= unsigned(hi - lo) || u < sink ||
           unsigned(u - blo) < unsigned(bhi - blo);
  }
};

// ----------------------------------------------------------------------------
// log-sum-exp combine of the key splits of one row block (rows [rlo, rhi))
// ----------------------------------------------------------------------------

template <typename T, int D>
__device__ inline void merge_rows(const MergeGroup& mg, int rlo, int rhi, const void* part_o,
                                  const float* part_lse, int RB, int Hq, int G, int S,
                                  void* out, float* lse, int tid, int nthr) {
  constexpr int TPR = D / 4;
  for (int idx = tid; idx < (rhi - rlo) * TPR; idx += nthr) {
    const int rloc = rlo + idx / TPR;
    const int d = 4 * (idx % TPR);
    const float* pl = part_lse + size_t(mg.part0) * RB + rloc;
    const T* po = static_cast<const T*>(part_o) + (size_t(mg.part0) * RB + rloc) * D + d;
    float mx = kNegInf;
#pragma unroll 8
    for (int i = 0; i < mg.nsplit; ++i) mx = fmaxf(mx, pl[size_t(i) * RB]);
    float z = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
    for (int i = 0; i < mg.nsplit; ++i) {
      const float li = pl[size_t(i) * RB];
      const float w = (li == kNegInf) ? 0.f : __expf(li - mx);
      float4 v;
      if constexpr (sizeof(T) == 4) {
        v = *reinterpret_cast<const float4*>(po + size_t(i) * RB * D);
      } else {
        const uint2 u = *reinterpret_cast<const uint2*>(po + size_t(i) * RB * D);
        v = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                        __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
      }
      z += w;
      acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
    }
    const float inv = z > 0.f ? 1.f / z : 0.f;
    const int r = mg.row0 + rloc;
    const int t = r / G, h = mg.g * G + r % G;
    T* orow = static_cast<T*>(out) + ((size_t(mg.b) * S + t) * Hq + h) * D;
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4*>(orow + d) =
          make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
    } else {
      uint2 u;
      u.x = pack_bf16(acc.x * inv, acc.y * inv);
      u.y = pack_bf16(acc.z * inv, acc.w * inv);
      *reinterpret_cast<uint2*>(orow + d) = u;
    }
    if (lse && d == 0) lse[(size_t(mg.b) * Hq + h) * S + t] = z > 0.f ? mx + __logf(z) : kNegInf;
  }
}

// ----------------------------------------------------------------------------
// attention
// ----------------------------------------------------------------------------

// Loads key tiles of one workgroup through registers into LDS.  Slot indices
// are fetched two tiles ahead of use and row data one tile ahead; `commit`
// turns keys to their final positions (decoding int8 first) and writes them row
// by row into sK[KT][LDK], and writes values transposed into sV[D][LDV].
// Cached tiles come from the pool (gather) or from pages; suffix tiles from
// k_suf / v_suf, with RoPE at span_end + u.
template <typename T, int D, int SRC, int NT>
struct TileLoader {
  using PoolT = typename std::conditional<SRC == SRC_POOL_I8, int8_t, T>::type;
  static constexpr bool kPaged = SRC == SRC_PAGED || SRC == SRC_PAGED_SIF;
  using Sh = Shape<T, PoolT, D, NT, kPaged>;
  using L = Lds<T, D>;
  static constexpr int HALF = D / 2;
  static constexpr int KUPK = D / 16;       // key units per key

  const AttnParams& a;
  const int tid, b, g, S, slot0, N, nct, page0;
  const int kp2;                            // first of the two keys of this thread's value units
  const T* ksuf;
  const T* vsuf;
  const PoolT* kpool;
  const PoolT* vpool;

  uint32_t rk[Sh::RKW], rv[Sh::RVW];
  uint32_t rk2[Sh::RKW], rv2[Sh::RVW];      // paged: a second tile in flight
  float ck[Sh::NKU][8], sk[Sh::NKU][8];     // cos/sin of this thread's key units
  int cs_seg[Sh::NKU];                      // segment the pool cos/sin belong to
  int2 nk[Sh::NKU];                         // (row, segment) of the next tile's keys
  int nv[2];                                // pool rows of its values (only the row: a
                                            // loaded word left unused would be reused
                                            // while its load is in flight)
  uint32_t kofs[Sh::NPK], vofs[Sh::NPV];    // paged: byte offsets of this thread's vectors
  float k_scale[Sh::NKU], v_scale[2];

  __device__ __forceinline__ TileLoader(const AttnParams& a_, int tid_, int b_, int g_, int slot0_,
                                        int N_, int page0_)
      : a(a_), tid(tid_), b(b_), g(g_), S(a_.S), slot0(slot0_), N(N_), nct((N_ + KT - 1) / KT),
        page0(page0_),
        kp2(2 * (tid_ % (KT / 2))), ksuf(static_cast<const T*>(a_.k_suf)),
        vsuf(static_cast<const T*>(a_.v_suf)), kpool(static_cast<const PoolT*>(a_.k)),
        vpool(static_cast<const PoolT*>(a_.v)) {
#pragma unroll
    for (int i = 0; i < Sh::NKU; ++i) {
      nk[i] = make_int2(0, -1);
      cs_seg[i] = -1;
      k_scale[i] = 1.f;
    }
    nv[0] = nv[1] = 0;
    if constexpr (kPaged) {
      constexpr int EPV = Sh::EPV;
#pragma unroll
      for (int i = 0; i < Sh::NPK; ++i) {
        const int u = tid + i * NT;
        kofs[i] = uint32_t((u / (D / EPV)) * D + (u % (D / EPV)) * EPV) * sizeof(T);
      }
#pragma unroll
      for (int i = 0; i < Sh::NPV; ++i) {
        const int u = tid + i * NT;
        vofs[i] = uint32_t((u / (KT / EPV)) * a.PS + (u % (KT / EPV)) * EPV) * sizeof(T);
      }
    }
    v_scale[0] = v_scale[1] = 1.f;
  }

  // Every load here and in fetch_data is unconditional, from a clamped index
  // inside the tile: a load whose destination was first set to a default would
  // make the compiler wait for all loads in flight, including the row loads of
  // the tile after next.  Past a partial tile's end the keys and values are
  // therefore copies of its last row (finite); the mask takes those keys' scores
  // to -inf, so their probabilities are exactly zero and nothing is zeroed.
  // SUF: the tile is a suffix tile (tile >= nct), known at compile time so
  // that a loop runs one kind of tile and its loads have one set of registers.
  template <bool SUF>
  __device__ __forceinline__ void fetch_idx(int tile) {
    if constexpr (SUF) return;              // suffix tiles need no index
    const int k0 = tile * KT;
    const int nvalid = min(KT, N - k0);     // >= 1 for a cached tile
    if constexpr (kPaged) {
      // a request's pages are consecutive: the page is page0 + k0 / PS, no table
      // read (a scalar load in flight would turn every LDS operand wait of the
      // tile into a full wait)
    } else {
#pragma unroll
      for (int i = 0; i < Sh::NKU; ++i) {
        const int u = tid + i * NT;
        const int kk = u / KUPK;
        nk[i] = a.slot_info[slot0 + k0 + min(kk, nvalid - 1)];
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        nv[j] = a.slot_info[slot0 + k0 + min(kp2 + j, nvalid - 1)].x;
      }
    }
  }

  // Paged tiles: buffer loads whose descriptors are this tile's key block and
  // transposed value block (scalar arithmetic); the per-thread offsets never
  // change.  Rows or columns past nvalid are read as they lie in the page
  // (keys are masked, values zeroed at commit); nothing outside the tile is read.
  // With `real` false the descriptors have no extent: the loads return zeros and
  // touch no memory, but still count, so a loop issues the same loads each turn.
  __device__ __forceinline__ void paged_fetch(int k0, uint32_t (&K)[Sh::RKW],
                                              uint32_t (&V)[Sh::RVW], bool real = true) {
    // page of the tile: tile / tiles-per-page as a multiply-high by a reciprocal
    // computed on the host (exact for the tile counts the plan admits)
    const unsigned tile = unsigned(k0) / KT;
    const unsigned prel = a.tpp == 1 ? tile : __umulhi(tile, a.tpp_magic);
    const size_t ph = size_t(page0 + int(prel)) * a.Hkv + g;
    const int off = int(tile - prel * unsigned(a.tpp)) * KT;
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(static_cast<const T*>(a.k) + (ph * a.PS + off) * D), 0,
        real ? KT * D * int(sizeof(T)) : 0, kBufferFlags);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(static_cast<const T*>(a.v) + ph * D * a.PS + off), 0,
        real ? ((D - 1) * a.PS + KT) * int(sizeof(T)) : 0, kBufferFlags);
    static_assert(Sh::PK_TOT % NT == 0 && Sh::PV_TOT % NT == 0,
                  "every thread loads whole page vectors");
#pragma unroll
    for (int i = 0; i < Sh::NPK; ++i) {
      const auto val = __builtin_amdgcn_raw_buffer_load_b128(kr, kofs[i], 0, 0);
      K[4 * i] = val[0]; K[4 * i + 1] = val[1]; K[4 * i + 2] = val[2]; K[4 * i + 3] = val[3];
    }
#pragma unroll
    for (int i = 0; i < Sh::NPV; ++i) {
      const auto val = __builtin_amdgcn_raw_buffer_load_b128(vr, vofs[i], 0, 0);
      V[4 * i] = val[0]; V[4 * i + 1] = val[1]; V[4 * i + 2] = val[2]; V[4 * i + 3] = val[3];
    }
  }
  __device__ __forceinline__ void paged_commit(int k0, const uint32_t (&K)[Sh::RKW],
                                               const uint32_t (&V)[Sh::RVW], T* sK, T* sV) {
    constexpr int EPV = Sh::EPV;
    const int nvalid = min(KT, N - k0);
#pragma unroll
    for (int i = 0; i < Sh::NPK; ++i) {
      const int u = tid + i * NT;
      const int kk = u / (D / EPV), vec = u % (D / EPV);
      *reinterpret_cast<uint4*>(sK + kk * L::LDK + vec * EPV) =
          make_uint4(K[4 * i], K[4 * i + 1], K[4 * i + 2], K[4 * i + 3]);
    }
#pragma unroll
    for (int i = 0; i < Sh::NPV; ++i) {
      const int u = tid + i * NT;
      const int d = u / (KT / EPV), vec = u % (KT / EPV);
      uint4 val = make_uint4(V[4 * i], V[4 * i + 1], V[4 * i + 2], V[4 * i + 3]);
      if (nvalid < KT) {                    // a partial tile (uniform): zero past its end
        if (vec * EPV + EPV > nvalid) val = keep_first<T>(val, nvalid - vec * EPV);
      }
      // the vector's two 8-byte halves (bf16: keys 8 vec + 0..3 and + 4..7), each to
      // its column
      T* row = sV + d * L::LDV;
      *reinterpret_cast<uint2*>(row + L::vcol(vec * EPV)) = make_uint2(val.x, val.y);
      *reinterpret_cast<uint2*>(row + L::vcol(vec * EPV + EPV / 2)) = make_uint2(val.z, val.w);
    }
  }
  // cached paged tile `tile` into / out of register set B
  template <int B>
  __device__ __forceinline__ void fetch_set(int tile, bool real) {
    if constexpr (B == 0) paged_fetch(tile * KT, rk, rv, real);
    else paged_fetch(tile * KT, rk2, rv2, real);
  }
  template <int B>
  __device__ __forceinline__ void commit_set(int tile, T* sK, T* sV) {
    if constexpr (B == 0) paged_commit(tile * KT, rk, rv, sK, sV);
    else paged_commit(tile * KT, rk2, rv2, sK, sV);
  }

  template <bool SUF>
  __device__ __forceinline__ void fetch_data(int tile) {
    const int k0 = SUF ? (tile - nct) * KT : tile * KT;
    const int nvalid = SUF ? min(KT, S - k0) : min(KT, N - k0);   // >= 1
    if constexpr (SUF) {
#pragma unroll
      for (int i = 0; i < Sh::NKU; ++i) {
        const int u = tid + i * NT;
        const int kk = u / KUPK, c = u % KUPK;
        uint32_t* w = rk + i * 2 * Sh::WA;
        if (Sh::KU_ALL || u < Sh::KU_TOT) {   // uniform per wavefront
          const size_t tok = size_t(b) * S + k0 + min(kk, nvalid - 1);
          const size_t row = tok * a.Hkv + g;
          raw_load8<T>(w, ksuf + row * D + 8 * c);
          raw_load8<T>(w + Sh::WA, ksuf + row * D + 8 * c + HALF);
          load_cs8(a.suf_cs + tok * HALF + 8 * c, ck[i], sk[i]);
          cs_seg[i] = -1;                     // not a pool segment's cos/sin
        }
      }
#pragma unroll
      for (int i = 0; i < Sh::NVU; ++i) {
        const int u = tid + i * NT;
        const int c = u / (KT / 2);
        uint32_t* w = rv + i * 2 * Sh::WA;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (Sh::VU_ALL || u < Sh::VU_TOT) {
            const size_t row = (size_t(b) * S + k0 + min(kp2 + j, nvalid - 1)) * a.Hkv + g;
            raw_load8<T>(w + j * Sh::WA, vsuf + row * D + 8 * c);
          }
        }
      }
    } else if constexpr (kPaged) {
      paged_fetch(k0, rk, rv);
    } else {
      // values, then keys, then the keys' cos/sin, which are loaded only where a
      // key unit's segment changes: the compiler's count of the loads in flight
      // is exact up to such a load and conservative after it, so the rows it
      // follows are not made to wait for each other
#pragma unroll
      for (int i = 0; i < Sh::NVU; ++i) {
        const int u = tid + i * NT;
        const int c = u / (KT / 2);
        uint32_t* w = rv + i * 2 * Sh::WP;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (Sh::VU_ALL || u < Sh::VU_TOT) {
            const size_t row = size_t(nv[j]) * a.Hkv + g;
            raw_load8<PoolT>(w + j * Sh::WP, vpool + row * D + 8 * c);
            if constexpr (SRC == SRC_POOL_I8) v_scale[j] = a.v_scale[row];
          }
        }
      }
#pragma unroll
      for (int i = 0; i < Sh::NKU; ++i) {
        const int u = tid + i * NT;
        const int c = u % KUPK;
        uint32_t* w = rk + i * 2 * Sh::WP;
        if (Sh::KU_ALL || u < Sh::KU_TOT) {
          const size_t row = size_t(nk[i].x) * a.Hkv + g;
          raw_load8<PoolT>(w, kpool + row * D + 8 * c);
          raw_load8<PoolT>(w + Sh::WP, kpool + row * D + 8 * c + HALF);
          if constexpr (SRC == SRC_POOL_I8) k_scale[i] = a.k_scale[row];
        }
      }
#pragma unroll
      for (int i = 0; i < Sh::NKU; ++i) {
        const int u = tid + i * NT;
        const int c = u % KUPK;
        if ((Sh::KU_ALL || u < Sh::KU_TOT) && nk[i].y != cs_seg[i]) {   // a segment's cos/sin stay until it changes
          load_cs8(a.seg_cs + size_t(nk[i].y) * HALF + 8 * c, ck[i], sk[i]);
          cs_seg[i] = nk[i].y;
        }
      }
    }
  }

  template <bool SUF>
  __device__ __forceinline__ void commit(int tile, T* sK, T* sV) {
    const int k0 = SUF ? (tile - nct) * KT : tile * KT;
    const int nvalid = SUF ? min(KT, S - k0) : min(KT, N - k0);
    if (SUF || !kPaged) {
      constexpr bool from_pool = !SUF;
#pragma unroll
      for (int i = 0; i < Sh::NKU; ++i) {
        const int u = tid + i * NT;
        if (!Sh::KU_ALL && u >= Sh::KU_TOT) continue;
        const int kk = u / KUPK, c = u % KUPK;
        T* dst = sK + kk * L::LDK + 8 * c;
        float x[8], y[8];
        if (from_pool) {
          if constexpr (!kPaged) {
            const uint32_t* w = rk + i * 2 * Sh::WP;
            raw_to_f8<PoolT>(w, x);
            raw_to_f8<PoolT>(w + Sh::WP, y);
            if constexpr (SRC == SRC_POOL_I8) {
#pragma unroll
              for (int e = 0; e < 8; ++e) { x[e] *= k_scale[i]; y[e] *= k_scale[i]; }
            }
          }
        } else {
          const uint32_t* w = rk + i * 2 * Sh::WA;
          raw_to_f8<T>(w, x);
          raw_to_f8<T>(w + Sh::WA, y);
        }
        rotate8(x, y, ck[i], sk[i]);
        store8(dst, x);
        store8(dst + HALF, y);
      }
#pragma unroll
      for (int i = 0; i < Sh::NVU; ++i) {
        const int u = tid + i * NT;
        if (!Sh::VU_ALL && u >= Sh::VU_TOT) continue;
        const int c = u / (KT / 2);
        // bf16 values that need no decode: a transposed word holds element e of
        // the two keys kp2 and kp2 + 1, i.e. one 16-bit half of each row's word
        constexpr bool kRawV = sizeof(T) == 2 && !(from_pool && SRC == SRC_POOL_I8);
        if (kRawV) {
          const uint32_t* w0 = rv + i * 2 * (from_pool ? Sh::WP : Sh::WA);
          const uint32_t* w1 = w0 + (from_pool ? Sh::WP : Sh::WA);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            T* dst = sV + (8 * c + e) * L::LDV + L::vcol(kp2);
            *reinterpret_cast<uint32_t*>(dst) =
                __builtin_amdgcn_perm(w1[e / 2], w0[e / 2], (e & 1) ? 0x07060302u : 0x05040100u);
          }
          continue;
        }
        float x0[8], x1[8];
        if (from_pool) {
          if constexpr (!kPaged) {
            const uint32_t* w = rv + i * 2 * Sh::WP;
            raw_to_f8<PoolT>(w, x0);
            raw_to_f8<PoolT>(w + Sh::WP, x1);
            if constexpr (SRC == SRC_POOL_I8) {
#pragma unroll
              for (int e = 0; e < 8; ++e) { x0[e] *= v_scale[0]; x1[e] *= v_scale[1]; }
            }
          }
        } else {
          const uint32_t* w = rv + i * 2 * Sh::WA;
          raw_to_f8<T>(w, x0);
          raw_to_f8<T>(w + Sh::WA, x1);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float a0 = x0[e], a1 = x1[e];
          T* dst = sV + (8 * c + e) * L::LDV + L::vcol(kp2);
          if constexpr (sizeof(T) == 2) {
            *reinterpret_cast<uint32_t*>(dst) = pack_bf16(a0, a1);
          } else {
            *reinterpret_cast<float2*>(dst) = make_float2(a0, a1);
          }
        }
      }
    } else {
      paged_commit(k0, rk, rv, sK, sV);
    }
  }
};

// One workgroup = NT / 64 wavefronts.  With KG = 1 each wavefront owns 32 query
// rows (256 per 512-thread workgroup) and every key of a tile; with KG = 2 row
// groups of 32 rows (128 rows per 512 threads, 64 per 256) each see one half of
// every 64-key tile, keep their own online softmax, and the two halves are
// combined through LDS at the end.  256-thread workgroups (64-row blocks) run two
// to a CU, so that two work items' latencies overlap.
template <typename T, int D, int SRC, int KG, int NT>
__global__ __launch_bounds__(NT, 2) void attn_kernel(AttnParams a) {
  constexpr int NRG = NT / 64 / KG;         // row groups
  constexpr int NKB = 2 / KG;               // 32-key blocks per wavefront and tile
  using M = Mma<T>;
  using Op = typename M::Op;
  using L = Lds<T, D>;
  using PoolT = typename std::conditional<SRC == SRC_POOL_I8, int8_t, T>::type;
  constexpr bool kPaged = SRC == SRC_PAGED || SRC == SRC_PAGED_SIF;
  constexpr bool kSif = SRC == SRC_PAGED_SIF;
  using Sh = Shape<T, PoolT, D, NT, kPaged>;
  constexpr int KPL = M::KPL;
  constexpr int KSTEP = 2 * KPL;            // contraction length of one MFMA
  constexpr int NQC = D / KSTEP;            // Q operand chunks over d
  constexpr int NDB = D / 32;               // 32-wide d blocks of the output
  constexpr int CPB = 32 / KSTEP;           // P*V chunks per 32-key block
  constexpr int NPC = KT / KSTEP;           // P*V chunks per key tile
  constexpr int HALF = D / 2;
  constexpr int KUPK = D / 16;              // key units per key

  // two stages of [keys | transposed values]
  constexpr int SBUF = 2 * L::TILE;
  __shared__ __attribute__((aligned(16))) T sbuf[SBUF];
  __shared__ int s_last;
  auto kst = [&](int i) { return sbuf + i * L::TILE; };
  auto vst = [&](int i) { return sbuf + i * L::TILE + KT * L::LDK; };

  const int tid = threadIdx.x;
  const WorkItem it = a.items[blockIdx.x];
  const int wave = tid >> 6, lane = tid & 63;
  const int qi = lane & 31, half = lane >> 5;
  const int b = it.b, g = it.g;
  const int S = a.S, G = a.G;
  const int slot0 = it.slot0;
  const int N = it.nslots;
  const int nct = (N + KT - 1) / KT;

  const int rgrp = wave % NRG, kh = wave / NRG;
  const int rloc = rgrp * 32 + qi;
  const bool row_ok = rloc < it.nrows;
  // a lane past the block's last row reads that row (its result is never
  // stored), so that every load is unconditional: a skipped load would leave
  // the compiler's wait counts conservative for everything issued before it
  const int r = it.row0 + min(rloc, it.nrows - 1);
  const int t = r / G;
  const int h = g * G + r % G;

  TileLoader<T, D, SRC, NT> ld(a, tid, b, g, slot0, N, it.page0);
  // suffix tiles (tile >= nct) and cached tiles run in loops of their own
  const int t0 = it.tile0, t1 = it.tile1;
  const int tc = min(t1, nct);             // cached tiles [t0, tc), suffix [max(t0, nct), t1)
  // tile at item position i: the identity, except for multi-range items of SIF
  // plans, whose positions run through up to three ranges of suffix tiles
  auto tile_of = [&](int i) -> int {
    if constexpr (kSif) {
      if (it.n_ranges > 0) {
#pragma unroll
        for (int r = 0; r < 3; ++r) {
          const int first = it.rng[r] & 0xffff, len = (it.rng[r] >> 16) - first;
          if (i < len) return first + i;
          i -= len;
        }
      }
    }
    return i;
  };

  // ---- Q operand: RoPE at span_end + t, softmax scale and log2(e) folded in.
  // Lane (qi, half) holds d = c*KSTEP + half*KPL + e in qop[c][e]; the RoPE
  // partner d + D/2 sits in chunk c + NQC/2 of the same lane.
  // The first key tile's slot indices and the Q and cos/sin loads are issued
  // first, then the tile's row loads (whose addresses wait only for the slot
  // indices), and only then is Q rotated, so the two latencies overlap.  The two kinds of first tile take
  // copies of their own: where both kinds' loads could precede one wait, the
  // compiler counts the other kind's loads in flight too.
  Op qop[NQC];
  auto q_prologue = [&](auto suf_c) __attribute__((always_inline)) {
    constexpr bool SUF = decltype(suf_c)::value;
    if constexpr (!SUF) ld.template fetch_idx<false>(t0);
    const T* qrow = static_cast<const T*>(a.q) + ((size_t(b) * S + t) * a.Hq + h) * D;
    const float2* cs = a.suf_cs + (size_t(b) * S + t) * HALF;
    constexpr int NW = KPL == 8 ? 4 : 1;                 // raw words per KPL elements
    uint32_t qx[NQC / 2][NW], qy[NQC / 2][NW];
    float qc[NQC / 2][KPL], qs[NQC / 2][KPL];
#pragma unroll
    for (int c = 0; c < NQC / 2; ++c) {
      const int d0 = c * KSTEP + half * KPL;
      if constexpr (KPL == 8) {
        raw_load8<T>(qx[c], qrow + d0);
        raw_load8<T>(qy[c], qrow + d0 + HALF);
        load_cs8(cs + d0, qc[c], qs[c]);
      } else {
        qx[c][0] = __float_as_uint(to_f(qrow[d0]));
        qy[c][0] = __float_as_uint(to_f(qrow[d0 + HALF]));
        const float2 w = cs[d0];
        qc[c][0] = w.x;
        qs[c][0] = w.y;
      }
    }
    ld.template fetch_data<SUF>(SUF ? tile_of(t0) : t0);
#pragma unroll
    for (int c = 0; c < NQC / 2; ++c) {
      float x[KPL], y[KPL];
      if constexpr (KPL == 8) {
        raw_to_f8<T>(qx[c], x);
        raw_to_f8<T>(qy[c], y);
      } else {
        x[0] = __uint_as_float(qx[c][0]);
        y[0] = __uint_as_float(qy[c][0]);
      }
#pragma unroll
      for (int e = 0; e < KPL; ++e) {
        rotate_pair(x[e], y[e], qc[c][e], qs[c][e]);
        x[e] *= a.qscale;
        y[e] *= a.qscale;
      }
      if constexpr (KPL == 1) {
        qop[c] = x[0];
        qop[c + NQC / 2] = y[0];
      } else {
#pragma unroll
        for (int e = 0; e < KPL; ++e) {
          qop[c][e] = from_f<T>(x[e]);
          qop[c + NQC / 2][e] = from_f<T>(y[e]);
        }
      }
    }
  };
  if (t0 < nct) q_prologue(std::false_type{});
  else q_prologue(std::true_type{});

  float m_run = kNegInf, l_run = 0.f;
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  // bf16: scores leave Q K^T already relative to the reference maximum, the
  // first MFMA of each chain adding `bias` (minus the reference, per row), so
  // the exponentials subtract nothing; the bias changes with the (lazy)
  // reference only.  m_biased: the reference it holds (0 while m_run is -inf).
  f32x16 bias;
#pragma unroll
  for (int v = 0; v < 16; ++v) bias[v] = 0.f;
  float m_biased = 0.f;

  // ---- S^T = K Q^T over this wavefront's 32-key blocks, accumulator lane = query
  auto qk = [&](const T* sK, f32x16 (&s)[NKB]) {
    if constexpr (KPL == 8 && kPaged) {
      // bf16 from pages: a ring of AH key fragments kept in flight ahead of
      // their MFMAs, the scheduling fences holding this issue order (measured a
      // little faster there, a little slower where the loader does more work)
      constexpr int NF = NKB * NQC, AH = 4;
      auto frag = [&](int f) {
        const int kb = kh * NKB + f / NQC;
        return *reinterpret_cast<const Op*>(sK + (kb * 32 + qi) * L::LDK + half * KPL +
                                            (f % NQC) * KSTEP);
      };
      Op kf[AH];
#pragma unroll
      for (int f = 0; f < AH; ++f) kf[f] = frag(f);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        // the first product of each chain takes the bias as its accumulator input
        s[f / NQC] = M::run(kf[f % AH], qop[f % NQC], f % NQC == 0 ? bias : s[f / NQC]);
        if (f + AH < NF) kf[f % AH] = frag(f + AH);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NKB; ++j) {
        const int kb = kh * NKB + j;
        if constexpr (KPL == 1) {
#pragma unroll
          for (int v = 0; v < 16; ++v) s[j][v] = 0.f;
        }
        const T* krow = sK + (kb * 32 + qi) * L::LDK + half * KPL;
#pragma unroll
        for (int c = 0; c < NQC; ++c) {
          Op ka;
          if constexpr (KPL == 1) ka = krow[c * KSTEP];
          else ka = *reinterpret_cast<const Op*>(krow + c * KSTEP);
          // bf16: the first product takes the bias as its accumulator input
          s[j] = M::run(ka, qop[c], (KPL == 8 && c == 0) ? bias : s[j]);
        }
      }
    }
  };

  // ---- causal / ragged-tail mask, then the new running maximum (base 2);
  // accumulator value v of block kb holds key 32*kb + 8*(v/4) + 4*half + v%4
  // (a tree of three-way maxima: a chain over the lane's 16 NKB scores would
  // leave every step waiting for the one before)
  auto max_of = [](const f32x16 (&s)[NKB]) {
    constexpr int N = 16 * NKB;
    float x[N];
#pragma unroll
    for (int j = 0; j < NKB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) x[16 * j + v] = s[j][v];
    int n = N;
#pragma unroll
    for (int lvl = 0; lvl < 4; ++lvl) {
      if (n == 1) break;
      int m = 0;
#pragma unroll
      for (int i = 0; i < N; i += 3) {
        if (i >= n) break;
        float r = x[i];
        if (i + 1 < n) r = fmaxf(r, x[i + 1]);
        if (i + 2 < n) r = fmaxf(r, x[i + 2]);
        x[m++] = r;
      }
      n = m;
    }
    return n == 1 ? x[0] : fmaxf(x[0], x[1]);
  };
  auto mask_max = [&](int tile, f32x16 (&s)[NKB]) {
    const bool suffix = tile >= nct;
    const int k0 = suffix ? (tile - nct) * KT : tile * KT;
    const int nvalid = suffix ? min(KT, S - k0) : min(KT, N - k0);
    if constexpr (kSif) {
      const RowKeys row_keys(t, a);
      // this wavefront's keys [w0, w1] lie in one of the row's visible ranges for
      // every lane (tiles below the causal diagonal): nothing to mask
      const int w0 = k0 + kh * NKB * 32, w1 = w0 + NKB * 32 - 1;
      const bool whole = nvalid == KT &&
                         ((w0 >= row_keys.lo && w1 <= row_keys.hi) || w1 < row_keys.sink ||
                          (w0 >= row_keys.blo && w1 < row_keys.bhi));
      if (!__all(whole)) {
        // the lane's visible keys among the wavefront's [w0, w0 + 32 NKB) as a bit
        // mask (bit k: key w0 + k), shifted so that accumulator value (j, v)
        // tests bit 32 j + 8 (v / 4) + v % 4, a constant: one bit-field extract and
        // one bit select per score
        auto bits = [](int x0, int x1) -> uint64_t {   // keys [x0, x1) relative to w0
          x0 = max(x0, 0);
          x1 = min(x1, 64);
          if (x1 <= x0) return 0;
          const uint64_t below1 = x1 == 64 ? ~0ull : (1ull << x1) - 1;
          return below1 & ~((1ull << x0) - 1);
        };
        uint64_t vis = bits(row_keys.lo - w0, row_keys.hi + 1 - w0) |
                       bits(-w0, row_keys.sink - w0) |
                       bits(row_keys.blo - w0, row_keys.bhi - w0);
        vis &= bits(0, nvalid - kh * NKB * 32);
        vis >>= 4 * half;
        const uint32_t hidden[2] = {~uint32_t(vis), ~uint32_t(vis >> 32)};
#pragma unroll
        for (int j = 0; j < NKB; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int off = 8 * (v >> 2) + (v & 3);        // bit in word j
            uint32_t x = __float_as_uint(s[j][v]), m;
            asm("v_bfe_i32 %1, %2, %3, 1\n\t"          // all ones where hidden
                "v_bfi_b32 %0, %1, %4, %0"
                : "+v"(x), "=&v"(m) : "v"(hidden[j]), "i"(off), "v"(0xff800000u));
            s[j][v] = __uint_as_float(x);
          }
      }
    } else if (suffix || nvalid < KT) {
      // key = base + off with off a constant per accumulator value, visible
      // where off <= lim.  In a suffix tile u <= t < S already implies
      // key < nvalid; a cached tile has no causal part.  A masked score's bits
      // are replaced by -inf's through the sign of lim - off (v_bfi_b32): no
      // compares, whose 64-bit lane masks the compiler kept live all at once,
      // spilling scalar registers into the key loop
      const int base = kh * NKB * 32 + 4 * half;
      const int lim = suffix ? t - k0 - base : nvalid - 1 - base;
      // (suffix tiles below the diagonal: every lane sees all its keys)
      if (!__all(lim >= 32 * (NKB - 1) + 27)) {
#pragma unroll
        for (int j = 0; j < NKB; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int off = j * 32 + 8 * (v >> 2) + (v & 3);
            uint32_t x = __float_as_uint(s[j][v]), m;
            asm("v_subrev_u32 %1, %3, %2\n\t"       // lim - off
                "v_ashrrev_i32 %1, 31, %1\n\t"      // all ones where masked
                "v_bfi_b32 %0, %1, %4, %0"
                : "+v"(x), "=&v"(m) : "v"(lim), "i"(off), "v"(0xff800000u));
            s[j][v] = __uint_as_float(x);
          }
      }
    }
    return fmaxf(m_run, half_pair_max(max_of(s)) + m_biased);   // absolute
  };

  // ---- rescale the running sum and output to a new maximum
  auto rescale = [&](float m_new, float m_ref) {
    if (__any(m_new > m_run)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    }
    m_run = m_new;
  };

  // ---- bf16: probabilities packed as P*V operands.  Chunk cc holds values
  // v0 + e, v0 = 8*(cc % 2), of block cc / 2; its row sum is taken from the
  // rounded values P*V uses
  constexpr int NPW = NPC / KG;           // P*V chunks per wavefront and tile
  auto exp_pack = [&](f32x16 (&s)[NKB], float m_ref, Op (&pb)[NPW]) {
    float psum = 0.f;
    if constexpr (KPL == 8) {
      // four independent partial sums, so that the dot products do not wait for
      // each other
      float ps[4] = {0.f, 0.f, 0.f, 0.f};
      const bf16x2 ones = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
#pragma unroll
      for (int cc = 0; cc < NPW; ++cc) {
        const int j = cc / CPB, v0 = KPL * (cc % CPB);
#pragma unroll
        for (int e = 0; e < KPL; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(s[j][v0 + e] - m_ref);
          const float p1 = __builtin_amdgcn_exp2f(s[j][v0 + e + 1] - m_ref);
          const f32x2 p01 = {p0, p1};
          const bf16x2 pp = __builtin_convertvector(p01, bf16x2);   // one paired conversion
          pb[cc][e] = pp[0];
          pb[cc][e + 1] = pp[1];
          ps[e / 2] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, ps[e / 2], false);
        }
      }
      psum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
    }
    return psum;
  };
  // ---- O^T += V^T P^T; chunk c of the tile covers keys 16*(c%2) + 4*half +
  // {0..3} and + 8 + {0..3} of block c / 2 (bf16: one 16-byte read at column
  // 16*(c%2) + 8*half of the block's permuted row)
  auto pv = [&](const T* sV, const Op (&pb)[NPW]) {
    if constexpr (KPL == 8 && kPaged) {
      // value fragments in a ring of AH ahead of their MFMAs, as for the keys
      constexpr int NF = NPW * NDB, AH = 4;
      auto frag = [&](int f) {
        const int cc = f / NDB, db = f % NDB;
        const int c = kh * NPW + cc;
        const T* vrow = sV + (db * 32 + qi) * L::LDV + (c / CPB) * 32 + 8 * half + 16 * (c % CPB);
        return *reinterpret_cast<const Op*>(vrow);
      };
      Op vf[AH];
#pragma unroll
      for (int f = 0; f < AH; ++f) vf[f] = frag(f);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        o[f % NDB] = M::run(vf[f % AH], pb[f / NDB], o[f % NDB]);
        if (f + AH < NF) vf[f % AH] = frag(f + AH);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else if constexpr (KPL == 8) {
#pragma unroll
      for (int cc = 0; cc < NPW; ++cc) {
        const int c = kh * NPW + cc;
        const int kb = c / CPB;
        const int kofs = 16 * (c % CPB);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const T* vrow = sV + (db * 32 + qi) * L::LDV + kb * 32 + 8 * half + kofs;
          o[db] = M::run(*reinterpret_cast<const Op*>(vrow), pb[cc], o[db]);
        }
      }
    }
  };

  // Tiles [ta, tb) of one kind.  Prologue: tile ta (its loads issued already
  // when `fetched`) into stage 0, tile ta + 1 in registers.  The loads of a
  // run's first tile cannot be issued under the previous run's last tile: a
  // load of the other kind anywhere in the loop would make the compiler's
  // waits there conservative again.
  // ---- one key tile in LDS stage `stage`: scores, online softmax, P*V
  auto tile_compute = [&](int tile, int stage) __attribute__((always_inline)) {
    f32x16 s[NKB];
    qk(kst(stage), s);
    const float m_new = mask_max(tile, s);
    const float m_ref = (m_new == kNegInf) ? 0.f : m_new;
    if constexpr (KPL == 8) {
      // bf16: the reference maximum moves only when some row's maximum outgrows it
      // by more than kLazyLog2 (a factor 2^kLazyLog2), so the output rescale is
      // rare; probabilities stay below 2^kLazyLog2, which bf16 and fp32 sums hold
      if (__any(m_new > m_run + kLazyLog2)) {
        rescale(m_new, m_ref);
        // re-base the scores and the bias on the new reference
        const float d = m_ref - m_biased;
#pragma unroll
        for (int j = 0; j < NKB; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) s[j][v] -= d;
#pragma unroll
        for (int v = 0; v < 16; ++v) bias[v] = -m_ref;
        m_biased = m_ref;
      }
      Op pb[NPW];
      l_run += exp_pack(s, 0.f, pb);
      pv(vst(stage), pb);
    } else {
      float psum = 0.f;
#pragma unroll
      for (int j = 0; j < NKB; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float p = __builtin_amdgcn_exp2f(s[j][v] - m_ref);
          s[j][v] = p;
          psum += p;
        }
      rescale(m_new, m_ref);
      l_run += psum;

      // ---- O^T += V^T P^T with fp32 MFMA: chunk c takes accumulator value
      // v0 = c % CPB of block c / CPB (key 8*(v0/4) + 4*half + v0%4 of it)
      const T* sV = vst(stage);
#pragma unroll
      for (int cc = 0; cc < NPC / KG; ++cc) {
        const int c = kh * (NPC / KG) + cc;
        const int j = cc / CPB;
        const int kb = c / CPB;
        const int v0 = KPL * (c % CPB);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const T* vrow = sV + (db * 32 + qi) * L::LDV + kb * 32 + 4 * half;
          o[db] = M::run(vrow[8 * (v0 >> 2) + (v0 & 3)], s[j][v0], o[db]);
        }
      }
    }
  };

  // in the paged loop below, a wavefront whose row group is empty (decode: 4
  // rows in a 128-row block) still loads and commits its share of each tile
  // but computes nothing
  const bool rows_here = rgrp * 32 < it.nrows;

  // bf16 pages with 512-thread workgroups keep two tiles' loads in flight, in two
  // register sets that alternate: for 128-row blocks (short suffixes, decode:
  // bandwidth-bound) and for 256-row blocks (long suffixes), where one tile of
  // compute did not cover the row loads' latency
  constexpr bool kDeep = kPaged && NT == 512 && sizeof(T) == 2;

  // Tiles [ta, tb) of one kind.  Prologue: tile ta (its loads issued already
  // when `fetched`) into stage 0, tile ta + 1 in registers.  The loads of a
  // run's first tile cannot be issued under the previous run's last tile: a
  // load of the other kind anywhere in the loop would make the compiler's
  // waits there conservative again.
  auto run_tiles = [&](auto suf_c, int ta, int tb, bool fetched) __attribute__((always_inline)) {
    constexpr bool SUF = decltype(suf_c)::value;
    if (ta >= tb) return;
    if constexpr (!SUF && kDeep) {
      // tile ta's loads are in set 0; tile t's set is (t - ta) & 1.  Every turn
      // issues its loads unconditionally (no-extent descriptors past the end),
      // so that the commits wait only for their own set.
      ld.template fetch_set<1>(ta + 1, ta + 1 < tb);
      ld.template commit_set<0>(ta, kst(0), vst(0));
      ld.template fetch_set<0>(ta + 2, ta + 2 < tb);
      __syncthreads();
      auto step = [&](auto nb_c, int tile) __attribute__((always_inline)) {
        constexpr int NB = decltype(nb_c)::value;   // register set of tile + 1
        const int stage = (tile - ta) & 1;
        if (tile + 1 < tb) ld.template commit_set<NB>(tile + 1, kst(stage ^ 1), vst(stage ^ 1));
        ld.template fetch_set<NB>(tile + 3, tile + 3 < tb);
        if (tile < tb && rows_here) tile_compute(tile, stage);
        __syncthreads();   // next stage written; this stage free for the tile after next
      };
      for (int tile = ta; tile < tb; tile += 2) {
        step(std::integral_constant<int, 1>{}, tile);
        step(std::integral_constant<int, 0>{}, tile + 1);
      }
    } else {
      // (positions i run through tiles tile_of(i))
      if (!fetched) ld.template fetch_data<SUF>(tile_of(ta));
      if (ta + 1 < tb) ld.template fetch_idx<SUF>(tile_of(ta + 1));
      ld.template commit<SUF>(tile_of(ta), kst(0), vst(0));
      if (ta + 1 < tb) ld.template fetch_data<SUF>(tile_of(ta + 1));
      if (ta + 2 < tb) ld.template fetch_idx<SUF>(tile_of(ta + 2));
      __syncthreads();
      for (int i = ta; i < tb; ++i) {
        const int stage = (i - ta) & 1;
        // next tile into the other stage; its readers finished before the last barrier
        if (i + 1 < tb) {
          ld.template commit<SUF>(tile_of(i + 1), kst(stage ^ 1), vst(stage ^ 1));
          if (i + 2 < tb) ld.template fetch_data<SUF>(tile_of(i + 2));
          if (i + 3 < tb) ld.template fetch_idx<SUF>(tile_of(i + 3));
        }
        tile_compute(tile_of(i), stage);
        __syncthreads();   // next stage written; this stage free for the tile after next
      }
    }
  };
  run_tiles(std::false_type{}, t0, tc, true);
  run_tiles(std::true_type{}, max(t0, nct), t1, t0 >= nct);

  // ---- the two key halves of a row group combine (same lane, same rows)
  if constexpr (KG == 2) {
    constexpr int XW = 2 + NDB * 16;                     // m, l and this lane's outputs
    static_assert(NRG * 64 * XW * sizeof(float) <= SBUF * sizeof(T),
                  "key-half exchange must fit in the tile stages");
    float* xs = reinterpret_cast<float*>(sbuf);          // [NRG][64 lanes][XW] floats
    float* mine = xs + (size_t(rgrp) * 64 + lane) * XW;
    if (kh == 1) {
      mine[0] = m_run;
      mine[1] = l_run;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) mine[2 + db * 16 + v] = o[db][v];
    }
    __syncthreads();
    if (kh == 0) {
      const float m1 = mine[0], l1 = mine[1];
      const float mx = fmaxf(m_run, m1);
      const float mr = (mx == kNegInf) ? 0.f : mx;
      const float a0 = __builtin_amdgcn_exp2f(m_run - mr), a1 = __builtin_amdgcn_exp2f(m1 - mr);
      l_run = l_run * a0 + l1 * a1;
      m_run = mx;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] = o[db][v] * a0 + mine[2 + db * 16 + v] * a1;
    }
  }
  const bool writer = KG == 1 || kh == 0;

  // ---- epilogue: rows normalised and staged in LDS (accumulator value v of
  // block db holds d = 32*db + 8*(v/4) + 4*half + v%4), then copied out as
  // whole rows: to the output, or in the activation dtype to the partials
  const float l_tot = half_pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_val = l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  constexpr int LDO = D + (sizeof(T) == 2 ? 4 : 2);   // staged row, 8-byte aligned
  static_assert(NRG * 32 * LDO <= SBUF, "staged rows must fit in the tile stages");
  if constexpr (KG == 2) __syncthreads();   // the key-half exchange is read before reuse
  if (writer) {
    T* srow = sbuf + (rgrp * 32 + qi) * LDO;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * db + 8 * i + 4 * half;
        const float x0 = o[db][4 * i] * inv, x1 = o[db][4 * i + 1] * inv;
        const float x2 = o[db][4 * i + 2] * inv, x3 = o[db][4 * i + 3] * inv;
        if constexpr (sizeof(T) == 4) {
          reinterpret_cast<float2*>(srow + d)[0] = make_float2(x0, x1);
          reinterpret_cast<float2*>(srow + d)[1] = make_float2(x2, x3);
        } else {
          *reinterpret_cast<uint2*>(srow + d) = make_uint2(pack_bf16(x0, x1), pack_bf16(x2, x3));
        }
      }
    if (row_ok && half == 0) {
      if (it.partial < 0) {
        if (a.lse) a.lse[(size_t(b) * a.Hq + h) * S + t] = lse_val;
      } else {
        a.part_lse[size_t(it.partial) * a.RB + rloc] = lse_val;
      }
    }
  }
  __syncthreads();
  {
    constexpr int EPC = 16 / int(sizeof(T));            // elements per 16-byte chunk
    constexpr int CPR = D / EPC;                         // chunks per row
    const int nrows = it.nrows;
    for (int ch = tid; ch < nrows * CPR; ch += NT) {
      const int rl = ch / CPR, e0 = (ch % CPR) * EPC;
      const T* src = sbuf + rl * LDO + e0;
      const uint2 lo = *reinterpret_cast<const uint2*>(src);
      const uint2 hi = *reinterpret_cast<const uint2*>(src + EPC / 2);
      T* dst;
      if (it.partial < 0) {
        const int r = it.row0 + rl;
        dst = static_cast<T*>(a.out) + ((size_t(b) * S + r / G) * a.Hq + g * G + r % G) * D + e0;
      } else {
        dst = static_cast<T*>(a.part_o) + (size_t(it.partial) * a.RB + rl) * D + e0;
      }
      *reinterpret_cast<uint4*>(dst) = make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
  }

  // ---- the last split of a row block to finish combines all of its splits
  if (it.merge >= 0 && a.merge_in_kernel) {
    // release this split's partial at agent scope (every wavefront: its stores are
    // written back past the L2 of its XCD before the barrier)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (tid == 0) {
      // system scope: the splits of a row block may run on different XCDs, whose
      // L2 caches are not coherent with each other; a system-scope atomic is
      // performed past them
      const int old = __hip_atomic_fetch_add(a.counters + it.merge, 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_SYSTEM);
      s_last = (old == a.merges[it.merge].nsplit - 1) ? 1 : 0;
    }
    __syncthreads();
    if (s_last) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // the other splits' partials
      const MergeGroup mg = a.merges[it.merge];
      merge_rows<T, D>(mg, 0, mg.nrows, a.part_o, a.part_lse, a.RB, a.Hq, G, S, a.out, a.lse,
                       tid, NT);
      if (tid == 0)                        // ready for the next launch
        __hip_atomic_store(a.counters + it.merge, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

// ----------------------------------------------------------------------------
// merge of key splits as its own kernel (row blocks with many splits)
// ----------------------------------------------------------------------------

// Rows of one merge group, RPW per workgroup, TPR threads per row with EPT
// output elements each.  The split LSEs and the partial rows of the first NB
// splits are loaded together (their addresses do not depend on each other),
// so that up to NB splits take one memory round trip; the LSEs are reduced
// across the row's threads into per-split weights in LDS.  Later batches of NB
// splits each take one more.  Partial rows are loaded only for the group's own
// splits (a branch uniform over the workgroup): clamped duplicates to fill a
// batch of 32 cost more than a second round trip.
template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeParams a) {
  constexpr int EPT = 4;
  constexpr int TPR = D / EPT;                 // threads per row
  constexpr int RPW = 256 / TPR;               // rows per workgroup
  constexpr int NPS = kMaxSplits / TPR;        // split LSEs per thread
  constexpr int NB = 32;                       // splits per batch of partial-row loads
  constexpr int WPE = EPT * sizeof(T) / 4;     // 32-bit words of a thread's elements
  __shared__ float s_w[kMaxSplits][RPW];
  const MergeGroup mg = a.groups[blockIdx.x];
  const int rlo = blockIdx.y * RPW;
  if (rlo >= mg.nrows) return;
  const int tid = threadIdx.x, rl = tid / TPR, sub = tid % TPR;
  const int rloc = rlo + rl;
  const bool ok = rloc < mg.nrows;
  const float* pl = a.part_lse + size_t(mg.part0) * a.RB + rloc;

  // LSE loads are unconditional, from indices clamped into the group's partials
  // (rows of a partial exist up to RB); what lies past the row count or the
  // split count gets weight zero.
  const int last = mg.nsplit - 1;
  float li[NPS];
#pragma unroll
  for (int k = 0; k < NPS; ++k) li[k] = pl[size_t(min(sub + k * TPR, last)) * a.RB];
  const T* po = static_cast<const T*>(a.part_o) + (size_t(mg.part0) * a.RB + rloc) * D + sub * EPT;
  uint32_t w[NB][WPE];                         // raw partial elements, decoded at use
  auto load_batch = [&](int i0) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      if (i0 + k > last) break;                // uniform: this group's splits only
      const uint32_t* src =
          reinterpret_cast<const uint32_t*>(po + size_t(i0 + k) * a.RB * D);
      if constexpr (WPE == 4) {
        const uint4 x = *reinterpret_cast<const uint4*>(src);
        w[k][0] = x.x; w[k][1] = x.y; w[k][2] = x.z; w[k][3] = x.w;
      } else {
        const uint2 x = *reinterpret_cast<const uint2*>(src);
        w[k][0] = x.x; w[k][1] = x.y;
      }
    }
  };
  load_batch(0);
  float mx = kNegInf;
#pragma unroll
  for (int k = 0; k < NPS; ++k) {
    if (!ok || sub + k * TPR > last) li[k] = kNegInf;
    mx = fmaxf(mx, li[k]);
  }
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  float z = 0.f;
#pragma unroll
  for (int k = 0; k < NPS; ++k) {
    const int i = sub + k * TPR;
    const float e = (li[k] == kNegInf) ? 0.f : __expf(li[k] - mx);
    if (i < mg.nsplit) s_w[i][rl] = e;
    z += e;
  }
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) z += __shfl_xor(z, off);
  __syncthreads();

  float acc[EPT] = {};
  for (int i0 = 0; i0 < mg.nsplit; i0 += NB) {
    if (i0 > 0) load_batch(i0);
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int i = i0 + k;
      if (i > last) break;                     // (its partial row was not loaded)
      const float wt = s_w[i][rl];
      float v[EPT];
      if constexpr (WPE == 4) {
#pragma unroll
        for (int e = 0; e < EPT; ++e) v[e] = __uint_as_float(w[k][e]);
      } else {
        v[0] = __uint_as_float(w[k][0] << 16);
        v[1] = __uint_as_float(w[k][0] & 0xffff0000u);
        v[2] = __uint_as_float(w[k][1] << 16);
        v[3] = __uint_as_float(w[k][1] & 0xffff0000u);
      }
#pragma unroll
      for (int e = 0; e < EPT; ++e) acc[e] += wt * v[e];
    }
  }
  if (!ok) return;
  const float inv = z > 0.f ? 1.f / z : 0.f;
  const int r = mg.row0 + rloc;
  const int t = r / a.G, h = mg.g * a.G + r % a.G;
  T* orow = static_cast<T*>(a.out) + ((size_t(mg.b) * a.S + t) * a.Hq + h) * D + sub * EPT;
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(orow) =
        make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  } else {
    *reinterpret_cast<uint2*>(orow) =
        make_uint2(pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv));
  }
  if (a.lse && sub == 0)
    a.lse[(size_t(mg.b) * a.Hq + h) * a.S + t] = z > 0.f ? mx + __logf(z) : kNegInf;
}

// One row per workgroup, the splits spread over SPL split lanes of TPR threads
// (row blocks with few rows and many splits: decode, short suffixes).  Each
// thread loads its first SPB splits' LSEs and partial elements together, so that
// up to SPL * SPB splits take one memory round trip; the maximum, the sum of
// weights and the weighted rows are reduced across lanes through LDS.  Later
// batches of SPB splits per lane each take one more.
template <typename T, int D>
__global__ __launch_bounds__(256) void merge_split_kernel(MergeParams a) {
  constexpr int EPT = 4;
  constexpr int TPR = D / EPT;                 // threads per row
  constexpr int SPL = 256 / TPR;               // split lanes
  constexpr int SPB = 8;                       // splits per lane per batch
  constexpr int WPE = EPT * sizeof(T) / 4;     // 32-bit words of a thread's elements
  __shared__ float s_red[256];
  __shared__ float s_acc[SPL][D];
  const MergeGroup mg = a.groups[blockIdx.x];
  const int rloc = blockIdx.y;
  if (rloc >= mg.nrows) return;
  const int tid = threadIdx.x, sl = tid / TPR, sub = tid % TPR;
  const int last = mg.nsplit - 1;
  const float* pl = a.part_lse + size_t(mg.part0) * a.RB + rloc;
  const T* po = static_cast<const T*>(a.part_o) + (size_t(mg.part0) * a.RB + rloc) * D + sub * EPT;

  // a batch: splits i0 + k * SPL, k < SPB, from indices clamped to the last
  // split (unconditional loads; what lies past it gets weight zero)
  float l[SPB];
  uint32_t w[SPB][WPE];
  auto load_batch = [&](int i0) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < SPB; ++k) {
      const int i = min(i0 + k * SPL, last);
      l[k] = pl[size_t(i) * a.RB];
      const uint32_t* src = reinterpret_cast<const uint32_t*>(po + size_t(i) * a.RB * D);
      if constexpr (WPE == 4) {
        const uint4 x = *reinterpret_cast<const uint4*>(src);
        w[k][0] = x.x; w[k][1] = x.y; w[k][2] = x.z; w[k][3] = x.w;
      } else {
        const uint2 x = *reinterpret_cast<const uint2*>(src);
        w[k][0] = x.x; w[k][1] = x.y;
      }
    }
  };
  load_batch(sl);

  // maximum over all split LSEs: the first batch's from registers, any later
  // batch's (LSEs only) read now
  float mx = kNegInf;
#pragma unroll
  for (int k = 0; k < SPB; ++k) mx = fmaxf(mx, sl + k * SPL <= last ? l[k] : kNegInf);
  for (int i0 = sl + SPL * SPB; i0 <= last; i0 += SPL * SPB) {
    float lk[SPB];
#pragma unroll
    for (int k = 0; k < SPB; ++k) lk[k] = pl[size_t(min(i0 + k * SPL, last)) * a.RB];
#pragma unroll
    for (int k = 0; k < SPB; ++k) mx = fmaxf(mx, i0 + k * SPL <= last ? lk[k] : kNegInf);
  }
  s_red[tid] = mx;
  __syncthreads();
  mx = kNegInf;
#pragma unroll 8
  for (int i = 0; i < 256; i += TPR) mx = fmaxf(mx, s_red[i]);
  __syncthreads();

  // weighted partial rows of this lane's splits
  float z = 0.f, acc[EPT] = {};
  for (int i0 = sl; i0 <= last; i0 += SPL * SPB) {
    if (i0 != sl) load_batch(i0);
#pragma unroll
    for (int k = 0; k < SPB; ++k) {
      const float wt = (i0 + k * SPL <= last && l[k] != kNegInf) ? __expf(l[k] - mx) : 0.f;
      float v[EPT];
      if constexpr (WPE == 4) {
#pragma unroll
        for (int e = 0; e < EPT; ++e) v[e] = __uint_as_float(w[k][e]);
      } else {
        v[0] = __uint_as_float(w[k][0] << 16);
        v[1] = __uint_as_float(w[k][0] & 0xffff0000u);
        v[2] = __uint_as_float(w[k][1] << 16);
        v[3] = __uint_as_float(w[k][1] & 0xffff0000u);
      }
      z += wt;
#pragma unroll
      for (int e = 0; e < EPT; ++e) acc[e] += wt * v[e];
    }
  }
  // lane sums: z from the sub == 0 thread of each lane, the rows element-wise
  s_red[tid] = z;
#pragma unroll
  for (int e = 0; e < EPT; ++e) s_acc[sl][sub * EPT + e] = acc[e];
  __syncthreads();
  if (sl != 0) return;
  float zt = 0.f;
#pragma unroll
  for (int j = 0; j < SPL; ++j) zt += s_red[j * TPR];
  float o[EPT] = {};
#pragma unroll
  for (int j = 0; j < SPL; ++j)
#pragma unroll
    for (int e = 0; e < EPT; ++e) o[e] += s_acc[j][sub * EPT + e];
  const float inv = zt > 0.f ? 1.f / zt : 0.f;
  const int r = mg.row0 + rloc;
  const int t = r / a.G, h = mg.g * a.G + r % a.G;
  T* orow = static_cast<T*>(a.out) + ((size_t(mg.b) * a.S + t) * a.Hq + h) * D + sub * EPT;
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(orow) = make_float4(o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
  } else {
    *reinterpret_cast<uint2*>(orow) =
        make_uint2(pack_bf16(o[0] * inv, o[1] * inv), pack_bf16(o[2] * inv, o[3] * inv));
  }
  if (a.lse && sub == 0)
    a.lse[(size_t(mg.b) * a.Hq + h) * a.S + t] = zt > 0.f ? mx + __logf(zt) : kNegInf;
}

// ----------------------------------------------------------------------------
// compose: gather -> decode -> turn -> paged write
// ----------------------------------------------------------------------------

// One workgroup per (key tile, kv-head).  Three phases, so that every load of
// a thread is in flight at once: the slot indices of its key and value units,
// then all rows and cos/sin, then the turned keys and the transposed values
// (through LDS) are written.  Loads are unconditional (indices clamped into the
// tile); keys and values past the tile's end are written as zeros.
template <typename T, int D, typename PoolT>
__global__ __launch_bounds__(256) void compose_kernel(ComposeParams a) {
  using L = Lds<T, D>;
  constexpr int NTH = 256;
  constexpr int KU = D / 16;                 // key units per key: 8-element pairs (c, c + D/2)
  constexpr int NKU = KT * KU / NTH;         // key units per thread
  constexpr int VU = D / 8;                  // value units per key: 8 elements
  constexpr int NVU = KT * VU / NTH;         // value units per thread (one key: tid % KT)
  static_assert(KT * KU % NTH == 0 && KT * VU % NTH == 0 && NTH % KT == 0,
                "every thread holds whole units of one value key");
  __shared__ __attribute__((aligned(16))) T sV[D * L::LDV];
  const int tid = threadIdx.x;
  const int4 tl = a.tiles[blockIdx.x];
  const int g = blockIdx.y;
  const int first = tl.x, nvalid = tl.y, off = tl.w;   // slots [first, first + nvalid)
  const size_t ph = size_t(tl.z) * a.Hkv + g;
  T* kpage = static_cast<T*>(a.k_pages) + (ph * a.PS + off) * D;
  T* vpage = static_cast<T*>(a.v_pages) + ph * D * a.PS + off;
  const PoolT* kpool = static_cast<const PoolT*>(a.k);
  const PoolT* vpool = static_cast<const PoolT*>(a.v);

  // ---- slot indices
  int2 ks[NKU];
  int kpos[NKU];
#pragma unroll
  for (int i = 0; i < NKU; ++i) {
    const int slot = first + min((tid + i * NTH) / KU, nvalid - 1);
    ks[i] = a.slot_info[slot];
    kpos[i] = a.out_pos ? a.slot_pos[slot] : 0;
  }
  const int vkk = tid % KT;
  const int vsrc = a.slot_info[first + min(vkk, nvalid - 1)].x;

  // ---- rows, scales and cos/sin
  float kx[NKU][8], ky[NKU][8], kc[NKU][8], kn[NKU][8], vx[NVU][8];
  float kscale[NKU], vscale = 1.f;
  const size_t vrow = size_t(vsrc) * a.Hkv + g;
#pragma unroll
  for (int i = 0; i < NVU; ++i) load8(vpool + vrow * D + 8 * ((tid + i * NTH) / KT), vx[i]);
  if constexpr (sizeof(PoolT) == 1) vscale = a.v_scale[vrow];
#pragma unroll
  for (int i = 0; i < NKU; ++i) {
    const int c = (tid + i * NTH) % KU;
    const size_t row = size_t(ks[i].x) * a.Hkv + g;
    load8(kpool + row * D + 8 * c, kx[i]);
    load8(kpool + row * D + 8 * c + D / 2, ky[i]);
    kscale[i] = 1.f;
    if constexpr (sizeof(PoolT) == 1) kscale[i] = a.k_scale[row];
    load_cs8(a.seg_cs + size_t(ks[i].y) * (D / 2) + 8 * c, kc[i], kn[i]);
  }

  // (a scheduling fence: left to itself the scheduler waits for the first
  // unit's rows before issuing the rest, to save registers)
  __builtin_amdgcn_sched_barrier(0);

  // ---- keys: decoded, turned by delta, straight to the page.  Every unit is
  // computed, past the tile's end with a zero scale: a branch there would sink
  // loads into it, behind the others.
#pragma unroll
  for (int i = 0; i < NKU; ++i) {
    const int u = tid + i * NTH;
    const int kk = u / KU, c = u % KU;
    const bool ok = kk < nvalid;
    const float sc = ok ? kscale[i] : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) { kx[i][e] *= sc; ky[i][e] *= sc; }
    rotate8(kx[i], ky[i], kc[i], kn[i]);
    T* dst = kpage + size_t(kk) * D + 8 * c;
    store8(dst, kx[i]);
    store8(dst + D / 2, ky[i]);
    if (ok && g == 0 && c == 0) {
      const int slot = first + kk;
      if (a.out_src_row) a.out_src_row[slot] = ks[i].x;
      if (a.out_pos) a.out_pos[slot] = kpos[i];
    }
  }
  // ---- values: decoded, transposed through LDS, then each d-row of the page segment
  const bool vok = vkk < nvalid;
#pragma unroll
  for (int i = 0; i < NVU; ++i) {
    const int c = (tid + i * NTH) / KT;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      sV[(8 * c + e) * L::LDV + vkk] = from_f<T>(vok ? vx[i][e] * vscale : 0.f);
  }
  __syncthreads();
  constexpr int EPV = 16 / sizeof(T);
  constexpr int VV = KT / EPV;
  for (int u = tid; u < D * VV; u += NTH) {
    const int d = u / VV, vec = u % VV;
    const uint2* src = reinterpret_cast<const uint2*>(sV + d * L::LDV + vec * EPV);
    const uint2 lo = src[0], hi = src[1];     // LDS rows are 8-byte aligned
    *reinterpret_cast<uint4*>(vpage + size_t(d) * a.PS + vec * EPV) =
        make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}

// ----------------------------------------------------------------------------
// launchers
// ----------------------------------------------------------------------------

// ----------------------------------------------------------------------------
// static scratch of the allocation-free entry point
// ----------------------------------------------------------------------------

// One array per GPU (each device holds its own copy, at its own address, until
// the process ends).  Host code never passes the array's name to a kernel or a
// copy: in host code it is only a stand-in, so its device address is looked up.
static __device__ __align__(256) unsigned char scratch[C2KV_STATIC_SCRATCH_BYTES];

hipError_t static_scratch(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = a;
  }
  *out = addr[dev];
  return hipSuccess;
}

namespace {

// Launch `kernel(params)`.  With timing events, the dispatch packet itself
// stamps them at kernel start and end (hipExtLaunchKernel), the same
// timestamps a kernel trace reports.
template <typename P>
hipError_t launch(const void* kernel, dim3 grid, dim3 block, hipStream_t st, const P& params,
                  hipEvent_t ev0, hipEvent_t ev1) {
  void* args[] = {const_cast<P*>(&params)};
  if (ev0 || ev1) return hipExtLaunchKernel(kernel, grid, block, args, 0, st, ev0, ev1, 0);
  return hipLaunchKernel(kernel, grid, block, args, 0, st);
}

template <typename T>
const T* at(const void* base, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const uint8_t*>(base) + off);
}
template <typename T>
T* at_mut(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<uint8_t*>(base) + off);
}

template <typename T, int D, int SRC>
hipError_t launch_attn_t(const AttnParams& ap, int n_items, int rows, hipStream_t st,
                         hipEvent_t e0, hipEvent_t e1) {
  if (rows == 64)
    return launch(reinterpret_cast<const void*>(&attn_kernel<T, D, SRC, 2, 256>), dim3(n_items),
                  dim3(256), st, ap, e0, e1);
  const void* k = rows == 256 ? reinterpret_cast<const void*>(&attn_kernel<T, D, SRC, 1, 512>)
                              : reinterpret_cast<const void*>(&attn_kernel<T, D, SRC, 2, 512>);
  return launch(k, dim3(n_items), dim3(512), st, ap, e0, e1);
}

template <typename T, int SRC>
hipError_t launch_attn_d(int D, const AttnParams& ap, int n, int rows, hipStream_t st,
                         hipEvent_t e0, hipEvent_t e1) {
  return D == 64 ? launch_attn_t<T, 64, SRC>(ap, n, rows, st, e0, e1)
                 : launch_attn_t<T, 128, SRC>(ap, n, rows, st, e0, e1);
}

}  // namespace

hipError_t launch_attention(const Plan& p, void* ws, int src_kind, const void* k, const void* v,
                            const float* k_scale, const float* v_scale, const void* q,
                            const void* k_suf, const void* v_suf, void* out, float* lse,
                            hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  AttnParams ap{};
  ap.Hq = p.cfg.n_q_heads;
  ap.Hkv = p.cfg.n_kv_heads;
  ap.G = p.group;
  ap.S = p.suffix_len;
  ap.PS = p.page_size;
  ap.tpp = p.page_size / KT;
  ap.tpp_magic = ap.tpp > 1 ? unsigned((uint64_t(1) << 32) / uint64_t(ap.tpp)) + 1u : 0u;
  ap.max_pages = p.max_pages;
  ap.RB = p.rows_per_block;
  ap.n_seg = p.n_segments;
  ap.merge_in_kernel = p.merge_in_kernel ? 1 : 0;
  ap.sif_n = p.sif_n;
  ap.sif_block = p.sif_block;
  ap.sif_sink = p.sif_sink;
  ap.qscale = p.qscale_log2;
  ap.req_slot0 = at<int>(ws, p.ws.req_slot0);
  ap.slot_info = at<int2>(ws, p.ws.slot_info);
  ap.seg_cs = at<float2>(ws, p.ws.seg_cs);
  ap.suf_cs = at<float2>(ws, p.ws.suf_cs);
  ap.block_table = at<int>(ws, p.ws.block_table);
  ap.items = at<WorkItem>(ws, p.ws.items);
  ap.merges = at<MergeGroup>(ws, p.ws.merges);
  ap.counters = at_mut<int>(ws, p.ws.counters);
  ap.k = k;
  ap.v = v;
  ap.k_scale = k_scale;
  ap.v_scale = v_scale;
  ap.q = q;
  ap.k_suf = k_suf;
  ap.v_suf = v_suf;
  ap.out = out;
  ap.lse = lse;
  ap.part_o = at_mut<unsigned char>(ws, p.ws.part_o);
  ap.part_lse = at_mut<float>(ws, p.ws.part_lse);
  const int n = static_cast<int>(p.items.size());
  const int rows = p.rows_per_block;      // selects the row-block shape
  const int D = p.cfg.head_dim;
  // a SIF plan has no cached tiles: its kernels never read k / v, whatever they are
  if (p.sif_n > 0) {
    if (p.cfg.act_dtype == C2KV_F32)
      return launch_attn_d<float, SRC_PAGED_SIF>(D, ap, n, rows, st, e0, e1);
    return launch_attn_d<__bf16, SRC_PAGED_SIF>(D, ap, n, rows, st, e0, e1);
  }
  if (p.cfg.act_dtype == C2KV_F32) {
    if (src_kind == SRC_PAGED) return launch_attn_d<float, SRC_PAGED>(D, ap, n, rows, st, e0, e1);
    return launch_attn_d<float, SRC_POOL>(D, ap, n, rows, st, e0, e1);
  }
  if (src_kind == SRC_PAGED) return launch_attn_d<__bf16, SRC_PAGED>(D, ap, n, rows, st, e0, e1);
  if (src_kind == SRC_POOL) return launch_attn_d<__bf16, SRC_POOL>(D, ap, n, rows, st, e0, e1);
  return launch_attn_d<__bf16, SRC_POOL_I8>(D, ap, n, rows, st, e0, e1);
}

hipError_t launch_merge(const Plan& p, void* ws, void* out, float* lse, hipStream_t st,
                        hipEvent_t e0, hipEvent_t e1) {
  if (p.merges.empty() || p.merge_in_kernel) return hipSuccess;
  MergeParams mp{};
  mp.Hq = p.cfg.n_q_heads;
  mp.G = p.group;
  mp.S = p.suffix_len;
  mp.RB = p.rows_per_block;
  mp.groups = at<MergeGroup>(ws, p.ws.merges);
  mp.part_o = at<unsigned char>(ws, p.ws.part_o);
  mp.part_lse = at<float>(ws, p.ws.part_lse);
  mp.out = out;
  mp.lse = lse;
  const int D = p.cfg.head_dim;
  if (p.max_splits > kSplitMergeMin && p.rows_per_block <= 128) {
    // many splits over few rows: one workgroup per row, splits spread over lanes
    // (256-row blocks have rows enough to fill the machine with 8 rows a group)
    const dim3 grid(static_cast<unsigned>(p.merges.size()), p.rows_per_block);
    const void* k;
    if (p.cfg.act_dtype == C2KV_F32)
      k = D == 64 ? reinterpret_cast<const void*>(&merge_split_kernel<float, 64>)
                  : reinterpret_cast<const void*>(&merge_split_kernel<float, 128>);
    else
      k = D == 64 ? reinterpret_cast<const void*>(&merge_split_kernel<__bf16, 64>)
                  : reinterpret_cast<const void*>(&merge_split_kernel<__bf16, 128>);
    return launch(k, grid, dim3(256), st, mp, e0, e1);
  }
  const int rpw = 256 / (D / 4);
  const dim3 grid(static_cast<unsigned>(p.merges.size()), (p.rows_per_block + rpw - 1) / rpw);
  const void* k;
  if (p.cfg.act_dtype == C2KV_F32)
    k = D == 64 ? reinterpret_cast<const void*>(&merge_kernel<float, 64>)
                : reinterpret_cast<const void*>(&merge_kernel<float, 128>);
  else
    k = D == 64 ? reinterpret_cast<const void*>(&merge_kernel<__bf16, 64>)
                : reinterpret_cast<const void*>(&merge_kernel<__bf16, 128>);
  return launch(k, grid, dim3(256), st, mp, e0, e1);
}

hipError_t launch_compose(const Plan& p, void* ws, int pool_dtype, const void* k, const void* v,
                          const float* k_scale, const float* v_scale, void* k_pages,
                          void* v_pages, int64_t* out_src_row, int32_t* out_pos,
                          hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const int n_tiles = static_cast<int>(p.compose_tiles.size() / 4);
  if (n_tiles == 0) return hipSuccess;
  ComposeParams cp{};
  cp.Hkv = p.cfg.n_kv_heads;
  cp.PS = p.page_size;
  cp.slot_info = at<int2>(ws, p.ws.slot_info);
  cp.slot_pos = at<int>(ws, p.ws.slot_pos);
  cp.seg_cs = at<float2>(ws, p.ws.seg_cs);
  cp.tiles = at<int4>(ws, p.ws.compose_tiles);
  cp.k = k;
  cp.v = v;
  cp.k_scale = k_scale;
  cp.v_scale = v_scale;
  cp.k_pages = k_pages;
  cp.v_pages = v_pages;
  cp.out_src_row = out_src_row;
  cp.out_pos = out_pos;
  const dim3 grid(n_tiles, p.cfg.n_kv_heads);
  const int D = p.cfg.head_dim;
  const void* k_;
  if (p.cfg.act_dtype == C2KV_F32)
    k_ = D == 64 ? reinterpret_cast<const void*>(&compose_kernel<float, 64, float>)
                 : reinterpret_cast<const void*>(&compose_kernel<float, 128, float>);
  else if (pool_dtype == C2KV_I8)
    k_ = D == 64 ? reinterpret_cast<const void*>(&compose_kernel<__bf16, 64, int8_t>)
                 : reinterpret_cast<const void*>(&compose_kernel<__bf16, 128, int8_t>);
  else
    k_ = D == 64 ? reinterpret_cast<const void*>(&compose_kernel<__bf16, 64, __bf16>)
                 : reinterpret_cast<const void*>(&compose_kernel<__bf16, 128, __bf16>);
  return launch(k_, grid, dim3(256), st, cp, e0, e1);
}

}  // namespace c2kv

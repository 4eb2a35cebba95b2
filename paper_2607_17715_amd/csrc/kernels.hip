// HIP kernels of the compose-and-attend path for gfx950 (CDNA4).
//
//   compose_kernel   blender B (Section 2.2, Eq. 3; Section 3.2; Appendix C):
//                    gather kept rows -> decode (int8 * scale) -> turn keys by
//                    their segment's delta -> write pages (V transposed in-page)
//   attn_kernel      attention of the query tokens over [KV_total, x_q]
//                    (Eq. 4): suffix RoPE on load, MFMA S^T = K Q^T, online
//                    softmax in base 2, MFMA O^T = V^T P^T; keys come from the
//                    pages, or straight from the pool (gather/decode/turn fused)
//   merge_kernel     log-sum-exp combine of key splits
//
// MFMA use.  One wavefront owns 32 query rows.  Scores are computed transposed
// (keys x queries) so that in the 32x32 accumulator layout every lane holds one
// query's scores: the row max needs a single exchange between the two 32-lane
// halves, and the probabilities feed the P*V product from the lane that holds
// them.  The contraction index of P*V (the key) is permuted to follow that
// accumulator layout; V^T is read from LDS with the same permutation.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "plan.hpp"

namespace c2kv {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

constexpr int KT = kKeyTile;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLn2 = 0.693147180559945309f;

enum Src { SRC_PAGED = 0, SRC_POOL = 1, SRC_POOL_I8 = 2 };

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
__device__ inline uint32_t pack_bf16(float a, float b) {
  const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<__bf16>(a));
  const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<__bf16>(b));
  return lo | (hi << 16);
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

// ----------------------------------------------------------------------------
// parameters
// ----------------------------------------------------------------------------

struct AttnParams {
  int Hq, Hkv, G, S, PS, max_pages, RB;
  float qscale;                 // softmax scale * log2(e)
  const int* req_slot0;
  const int* slot_src;
  const int* slot_seg;
  const float2* seg_cs;
  const float2* suf_cs;
  const int* block_table;
  const WorkItem* items;
  const void* k;                // pages or pool
  const void* v;
  const float* k_scale;
  const float* v_scale;
  const void* q;
  const void* k_suf;
  const void* v_suf;
  void* out;
  float* lse;
  float* part_o;
  float* part_lse;
};

struct ComposeParams {
  int Hkv, PS, max_pages;
  const int* req_slot0;
  const int* slot_src;
  const int* slot_seg;
  const int* slot_pos;
  const float2* seg_cs;
  const int* block_table;
  const int* tiles;            // [n][2] (b, tile)
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
  const float* part_o;
  const float* part_lse;
  void* out;
  float* lse;
};

// ----------------------------------------------------------------------------
// tile loaders: fill sK[KT][D + pad] (keys at final positions) and
// sV[D][KT + pad] (values transposed); keys >= nvalid are zero-filled.
// ----------------------------------------------------------------------------

template <typename T, int D>
struct Lds {
  static constexpr int PAD = 16 / sizeof(T);
  static constexpr int LDK = D + PAD;
  static constexpr int LDV = KT + PAD;
};

// keys from one row per key (pool or suffix), turned by a per-key cos/sin row
// and decoded with an optional per-key scale; values transposed into sV.
template <typename T, int D, typename Src, typename RowFn>
__device__ inline void load_rows_tile(T* sK, T* sV, int nvalid, RowFn row_of) {
  using L = Lds<T, D>;
  constexpr int KU = D / 16;                // (chunk, chunk + D/2) pairs per key
  for (int u = threadIdx.x; u < KT * KU; u += blockDim.x) {
    const int kk = u / KU, c = u % KU;
    T* dst = sK + kk * L::LDK + 8 * c;
    if (kk < nvalid) {
      const Src* kp; const Src* vp; float ks, vs; const float2* cs;
      row_of(kk, kp, vp, ks, vs, cs);
      float x[8], y[8], cc[8], ss[8];
      load8(kp + 8 * c, x);
      load8(kp + 8 * c + D / 2, y);
      if constexpr (sizeof(Src) == 1) {
#pragma unroll
        for (int e = 0; e < 8; ++e) { x[e] *= ks; y[e] *= ks; }
      }
      load_cs8(cs + 8 * c, cc, ss);
      rotate8(x, y, cc, ss);
      store8(dst, x);
      store8(dst + D / 2, y);
    } else {
      store8_zero(dst);
      store8_zero(dst + D / 2);
    }
  }
  constexpr int VU = D / 8;                 // 8-element chunks per key
  for (int u = threadIdx.x; u < KT * VU; u += blockDim.x) {
    const int c = u / KT, kk = u % KT;
    float x[8];
    if (kk < nvalid) {
      const Src* kp; const Src* vp; float ks, vs; const float2* cs;
      row_of(kk, kp, vp, ks, vs, cs);
      load8(vp + 8 * c, x);
      if constexpr (sizeof(Src) == 1) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] *= vs;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sV[(8 * c + e) * L::LDV + kk] = from_f<T>(x[e]);
  }
}

// keys and transposed values straight from a page (already composed)
template <typename T, int D>
__device__ inline void load_paged_tile(T* sK, T* sV, const T* kpage, const T* vpage,
                                       int PS, int nvalid) {
  using L = Lds<T, D>;
  constexpr int EPV = 16 / sizeof(T);       // elements per 16-byte vector
  constexpr int KV = D / EPV;               // vectors per key row
  for (int u = threadIdx.x; u < KT * KV; u += blockDim.x) {
    const int kk = u / KV, vec = u % KV;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (kk < nvalid) val = *reinterpret_cast<const uint4*>(kpage + size_t(kk) * D + vec * EPV);
    *reinterpret_cast<uint4*>(sK + kk * L::LDK + vec * EPV) = val;
  }
  constexpr int VV = KT / EPV;              // vectors per transposed value row
  for (int u = threadIdx.x; u < D * VV; u += blockDim.x) {
    const int d = u / VV, vec = u % VV;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    const int k0 = vec * EPV;
    if (k0 + EPV <= nvalid) {
      val = *reinterpret_cast<const uint4*>(vpage + size_t(d) * PS + k0);
    } else if (k0 < nvalid) {
      T tmp[EPV];
#pragma unroll
      for (int e = 0; e < EPV; ++e) tmp[e] = (k0 + e < nvalid) ? vpage[size_t(d) * PS + k0 + e] : from_f<T>(0.f);
      val = *reinterpret_cast<const uint4*>(tmp);
    }
    *reinterpret_cast<uint4*>(sV + d * L::LDV + k0) = val;
  }
}

// ----------------------------------------------------------------------------
// attention
// ----------------------------------------------------------------------------

template <typename T, int D, int SRC>
__global__ __launch_bounds__(512) void attn_kernel(AttnParams a) {
  using M = Mma<T>;
  using Op = typename M::Op;
  using L = Lds<T, D>;
  using PoolT = typename std::conditional<SRC == SRC_POOL_I8, int8_t, T>::type;
  constexpr int KPL = M::KPL;
  constexpr int KSTEP = 2 * KPL;            // contraction length of one MFMA
  constexpr int NQC = D / KSTEP;            // Q operand chunks over d
  constexpr int NDB = D / 32;               // 32-wide d blocks of the output
  constexpr int CPB = 32 / KSTEP;           // P*V chunks per 32-key block
  constexpr int NPC = KT / KSTEP;           // P*V chunks per key tile

  __shared__ __attribute__((aligned(16))) T sK[KT * L::LDK];
  __shared__ __attribute__((aligned(16))) T sV[D * L::LDV];

  const WorkItem it = a.items[blockIdx.x];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int qi = lane & 31, half = lane >> 5;
  const int b = it.b, g = it.g;
  const int slot0 = a.req_slot0[b];
  const int N = a.req_slot0[b + 1] - slot0;
  const int nct = (N + KT - 1) / KT;
  const int S = a.S, G = a.G;

  const int rloc = wave * 32 + qi;
  const bool row_ok = rloc < it.nrows;
  const int r = it.row0 + rloc;
  const int t = row_ok ? r / G : 0;
  const int h = g * G + (row_ok ? r % G : 0);

  // ---- Q operand: RoPE at span_end + t, softmax scale and log2(e) folded in.
  // Lane (qi, half) holds d = c*KSTEP + half*KPL + e in qop[c][e]; the RoPE
  // partner d + D/2 sits in chunk c + NQC/2 of the same lane.
  Op qop[NQC];
  {
    const T* qrow = static_cast<const T*>(a.q) + ((size_t(b) * S + t) * a.Hq + h) * D;
    const float2* cs = a.suf_cs + (size_t(b) * S + t) * (D / 2);
#pragma unroll
    for (int c = 0; c < NQC / 2; ++c) {
#pragma unroll
      for (int e = 0; e < KPL; ++e) {
        const int d = c * KSTEP + half * KPL + e;
        float x = 0.f, y = 0.f;
        if (row_ok) {
          x = to_f(qrow[d]);
          y = to_f(qrow[d + D / 2]);
          const float2 w = cs[d];
          rotate_pair(x, y, w.x, w.y);
          x *= a.qscale;
          y *= a.qscale;
        }
        if constexpr (KPL == 1) {
          qop[c] = x;
          qop[c + NQC / 2] = y;
        } else {
          qop[c][e] = from_f<T>(x);
          qop[c + NQC / 2][e] = from_f<T>(y);
        }
      }
    }
  }

  float m_run = kNegInf, l_run = 0.f;
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;

  for (int tile = it.tile0; tile < it.tile1; ++tile) {
    const bool suffix = tile >= nct;
    const int k0 = suffix ? (tile - nct) * KT : tile * KT;
    const int nvalid = suffix ? min(KT, S - k0) : min(KT, N - k0);

    __syncthreads();   // previous tile fully consumed
    if (suffix) {
      const T* ksb = static_cast<const T*>(a.k_suf);
      const T* vsb = static_cast<const T*>(a.v_suf);
      load_rows_tile<T, D, T>(sK, sV, nvalid,
          [&](int kk, const T*& kp, const T*& vp, float& ks, float& vs, const float2*& cs) {
            const size_t row = (size_t(b) * S + k0 + kk) * a.Hkv + g;
            kp = ksb + row * D;
            vp = vsb + row * D;
            ks = vs = 1.f;
            cs = a.suf_cs + (size_t(b) * S + k0 + kk) * (D / 2);
          });
    } else if constexpr (SRC == SRC_PAGED) {
      const int page = a.block_table[size_t(b) * a.max_pages + k0 / a.PS];
      const int off = k0 % a.PS;
      const size_t ph = size_t(page) * a.Hkv + g;
      const T* kpage = static_cast<const T*>(a.k) + (ph * a.PS + off) * D;
      const T* vpage = static_cast<const T*>(a.v) + ph * D * a.PS + off;
      load_paged_tile<T, D>(sK, sV, kpage, vpage, a.PS, nvalid);
    } else {
      const PoolT* kpool = static_cast<const PoolT*>(a.k);
      const PoolT* vpool = static_cast<const PoolT*>(a.v);
      load_rows_tile<T, D, PoolT>(sK, sV, nvalid,
          [&](int kk, const PoolT*& kp, const PoolT*& vp, float& ks, float& vs,
              const float2*& cs) {
            const int slot = slot0 + k0 + kk;
            const size_t row = size_t(a.slot_src[slot]) * a.Hkv + g;
            kp = kpool + row * D;
            vp = vpool + row * D;
            if constexpr (SRC == SRC_POOL_I8) {
              ks = a.k_scale[row];
              vs = a.v_scale[row];
            } else {
              ks = vs = 1.f;
            }
            cs = a.seg_cs + size_t(a.slot_seg[slot]) * (D / 2);
          });
    }
    __syncthreads();

    // ---- S^T = K Q^T: two 32-key blocks, accumulator lane = query
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
      const T* krow = sK + (kb * 32 + qi) * L::LDK + half * KPL;
#pragma unroll
      for (int c = 0; c < NQC; ++c) {
        Op ka;
        if constexpr (KPL == 1) ka = krow[c * KSTEP];
        else ka = *reinterpret_cast<const Op*>(krow + c * KSTEP);
        s[kb] = M::run(ka, qop[c], s[kb]);
      }
    }

    // ---- mask and online softmax (base 2); accumulator value v of block kb
    // holds key 32*kb + 8*(v/4) + 4*half + v%4 of the tile
    float mt = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = kb * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
        const bool vis = key < nvalid && (!suffix || k0 + key <= t);
        const float x = vis ? s[kb][v] : kNegInf;
        s[kb][v] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float m_ref = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(s[kb][v] - m_ref);
        s[kb][v] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][v] *= alpha;

    // ---- O^T += V^T P^T.  Chunk c takes accumulator values
    // v = KPL*(c % CPB) + e of block c / CPB; the matching key is read from sV.
#pragma unroll
    for (int c = 0; c < NPC; ++c) {
      const int kb = c / CPB;
      const int v0 = KPL * (c % CPB);
      Op pb;
      if constexpr (KPL == 1) {
        pb = s[kb][v0];
      } else {
#pragma unroll
        for (int e = 0; e < KPL; ++e) pb[e] = from_f<T>(s[kb][v0 + e]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const T* vrow = sV + (db * 32 + qi) * L::LDV + kb * 32 + 4 * half;
        Op va;
        if constexpr (KPL == 1) {
          va = vrow[8 * (v0 >> 2) + (v0 & 3)];
        } else {
          // v0 = 8*(c%2): keys 16*(c%2) + 4*half + {0..3} and + 8 + {0..3}
          const int kofs = 8 * (v0 >> 2);
          const uint2 lo = *reinterpret_cast<const uint2*>(vrow + kofs);
          const uint2 hi = *reinterpret_cast<const uint2*>(vrow + kofs + 8);
          const uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
          va = __builtin_bit_cast(Op, u);
        }
        o[db] = M::run(va, pb, o[db]);
      }
    }
  }

  // ---- epilogue: accumulator value v of block db holds d = 32*db + 8*(v/4) + 4*half + v%4
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_val = l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  if (it.partial < 0) {
    T* orow = static_cast<T*>(a.out) + ((size_t(b) * S + t) * a.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * db + 8 * i + 4 * half;
        if constexpr (sizeof(T) == 4) {
          *reinterpret_cast<float4*>(orow + d) =
              make_float4(o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv,
                          o[db][4 * i + 3] * inv);
        } else {
          uint2 u;
          u.x = pack_bf16(o[db][4 * i] * inv, o[db][4 * i + 1] * inv);
          u.y = pack_bf16(o[db][4 * i + 2] * inv, o[db][4 * i + 3] * inv);
          *reinterpret_cast<uint2*>(orow + d) = u;
        }
      }
    if (a.lse && half == 0) a.lse[(size_t(b) * a.Hq + h) * S + t] = lse_val;
  } else {
    float* prow = a.part_o + (size_t(it.partial) * a.RB + rloc) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * db + 8 * i + 4 * half;
        *reinterpret_cast<float4*>(prow + d) =
            make_float4(o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv,
                        o[db][4 * i + 3] * inv);
      }
    if (half == 0) a.part_lse[size_t(it.partial) * a.RB + rloc] = lse_val;
  }
}

// ----------------------------------------------------------------------------
// merge of key splits
// ----------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeParams a) {
  constexpr int TPR = D / 4;                  // threads per row, 4 elements each
  constexpr int RPW = 256 / TPR;              // rows per workgroup
  const MergeGroup mg = a.groups[blockIdx.x];
  const int rloc = blockIdx.y * RPW + threadIdx.x / TPR;
  if (rloc >= mg.nrows) return;
  const int d = 4 * (threadIdx.x % TPR);
  float mx = kNegInf;
  for (int i = 0; i < mg.nsplit; ++i)
    mx = fmaxf(mx, a.part_lse[size_t(mg.part0 + i) * a.RB + rloc]);
  float z = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int i = 0; i < mg.nsplit; ++i) {
    const float li = a.part_lse[size_t(mg.part0 + i) * a.RB + rloc];
    const float w = (li == kNegInf) ? 0.f : __expf(li - mx);
    z += w;
    if (w != 0.f) {
      const float4 v = *reinterpret_cast<const float4*>(
          a.part_o + (size_t(mg.part0 + i) * a.RB + rloc) * D + d);
      acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
    }
  }
  const float inv = z > 0.f ? 1.f / z : 0.f;
  const int r = mg.row0 + rloc;
  const int t = r / a.G, h = mg.g * a.G + r % a.G;
  T* orow = static_cast<T*>(a.out) + ((size_t(mg.b) * a.S + t) * a.Hq + h) * D;
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(orow + d) =
        make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  } else {
    uint2 u;
    u.x = pack_bf16(acc.x * inv, acc.y * inv);
    u.y = pack_bf16(acc.z * inv, acc.w * inv);
    *reinterpret_cast<uint2*>(orow + d) = u;
  }
  if (a.lse && d == 0)
    a.lse[(size_t(mg.b) * a.Hq + h) * a.S + t] = z > 0.f ? mx + __logf(z) : kNegInf;
}

// ----------------------------------------------------------------------------
// compose: gather -> decode -> turn -> paged write
// ----------------------------------------------------------------------------

template <typename T, int D, typename PoolT>
__global__ __launch_bounds__(256) void compose_kernel(ComposeParams a) {
  using L = Lds<T, D>;
  __shared__ __attribute__((aligned(16))) T sV[D * L::LDV];
  const int b = a.tiles[2 * blockIdx.x], tile = a.tiles[2 * blockIdx.x + 1];
  const int g = blockIdx.y;
  const int slot0 = a.req_slot0[b];
  const int N = a.req_slot0[b + 1] - slot0;
  const int k0 = tile * KT;
  const int nvalid = min(KT, N - k0);
  const int page = a.block_table[size_t(b) * a.max_pages + k0 / a.PS];
  const int off = k0 % a.PS;
  const size_t ph = size_t(page) * a.Hkv + g;
  T* kpage = static_cast<T*>(a.k_pages) + (ph * a.PS + off) * D;
  T* vpage = static_cast<T*>(a.v_pages) + ph * D * a.PS + off;
  const PoolT* kpool = static_cast<const PoolT*>(a.k);
  const PoolT* vpool = static_cast<const PoolT*>(a.v);

  // keys: straight to the page, turned by delta
  constexpr int KU = D / 16;
  for (int u = threadIdx.x; u < KT * KU; u += blockDim.x) {
    const int kk = u / KU, c = u % KU;
    T* dst = kpage + size_t(kk) * D + 8 * c;
    if (kk < nvalid) {
      const int slot = slot0 + k0 + kk;
      const int src = a.slot_src[slot];
      const size_t row = size_t(src) * a.Hkv + g;
      float x[8], y[8], cc[8], ss[8];
      load8(kpool + row * D + 8 * c, x);
      load8(kpool + row * D + 8 * c + D / 2, y);
      if constexpr (sizeof(PoolT) == 1) {
        const float ks = a.k_scale[row];
#pragma unroll
        for (int e = 0; e < 8; ++e) { x[e] *= ks; y[e] *= ks; }
      }
      load_cs8(a.seg_cs + size_t(a.slot_seg[slot]) * (D / 2) + 8 * c, cc, ss);
      rotate8(x, y, cc, ss);
      store8(dst, x);
      store8(dst + D / 2, y);
      if (g == 0 && c == 0) {
        if (a.out_src_row) a.out_src_row[slot] = src;
        if (a.out_pos) a.out_pos[slot] = a.slot_pos[slot];
      }
    } else {
      store8_zero(dst);
      store8_zero(dst + D / 2);
    }
  }
  // values: transpose through LDS, then write each d-row of the page segment
  constexpr int VU = D / 8;
  for (int u = threadIdx.x; u < KT * VU; u += blockDim.x) {
    const int c = u / KT, kk = u % KT;
    float x[8];
    if (kk < nvalid) {
      const size_t row = size_t(a.slot_src[slot0 + k0 + kk]) * a.Hkv + g;
      load8(vpool + row * D + 8 * c, x);
      if constexpr (sizeof(PoolT) == 1) {
        const float vs = a.v_scale[row];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] *= vs;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sV[(8 * c + e) * L::LDV + kk] = from_f<T>(x[e]);
  }
  __syncthreads();
  constexpr int EPV = 16 / sizeof(T);
  constexpr int VV = KT / EPV;
  for (int u = threadIdx.x; u < D * VV; u += blockDim.x) {
    const int d = u / VV, vec = u % VV;
    *reinterpret_cast<uint4*>(vpage + size_t(d) * a.PS + vec * EPV) =
        *reinterpret_cast<const uint4*>(sV + d * L::LDV + vec * EPV);
  }
}

// ----------------------------------------------------------------------------
// launchers
// ----------------------------------------------------------------------------

namespace {

template <typename T>
const T* at(const void* base, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const uint8_t*>(base) + off);
}
template <typename T>
T* at_mut(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<uint8_t*>(base) + off);
}

template <typename T, int D, int SRC>
hipError_t launch_attn_t(const AttnParams& ap, int n_items, int threads, hipStream_t st) {
  hipLaunchKernelGGL((attn_kernel<T, D, SRC>), dim3(n_items), dim3(threads), 0, st, ap);
  return hipGetLastError();
}

template <typename T, int SRC>
hipError_t launch_attn_d(int D, const AttnParams& ap, int n, int threads, hipStream_t st) {
  return D == 64 ? launch_attn_t<T, 64, SRC>(ap, n, threads, st)
                 : launch_attn_t<T, 128, SRC>(ap, n, threads, st);
}

}  // namespace

hipError_t launch_attention(const Plan& p, int src_kind, const void* k, const void* v,
                            const float* k_scale, const float* v_scale, const void* q,
                            const void* k_suf, const void* v_suf, void* out, float* lse,
                            hipStream_t st) {
  const void* ws = p.d_workspace;
  AttnParams ap{};
  ap.Hq = p.cfg.n_q_heads;
  ap.Hkv = p.cfg.n_kv_heads;
  ap.G = p.group;
  ap.S = p.suffix_len;
  ap.PS = p.page_size;
  ap.max_pages = p.max_pages;
  ap.RB = p.rows_per_block;
  ap.qscale = p.qscale_log2;
  ap.req_slot0 = at<int>(ws, p.ws.req_slot0);
  ap.slot_src = at<int>(ws, p.ws.slot_src);
  ap.slot_seg = at<int>(ws, p.ws.slot_seg);
  ap.seg_cs = at<float2>(ws, p.ws.seg_cs);
  ap.suf_cs = at<float2>(ws, p.ws.suf_cs);
  ap.block_table = at<int>(ws, p.ws.block_table);
  ap.items = at<WorkItem>(ws, p.ws.items);
  ap.k = k;
  ap.v = v;
  ap.k_scale = k_scale;
  ap.v_scale = v_scale;
  ap.q = q;
  ap.k_suf = k_suf;
  ap.v_suf = v_suf;
  ap.out = out;
  ap.lse = lse;
  ap.part_o = at_mut<float>(p.d_workspace, p.ws.part_o);
  ap.part_lse = at_mut<float>(p.d_workspace, p.ws.part_lse);
  const int n = static_cast<int>(p.items.size());
  const int threads = 64 * (p.rows_per_block / kRowsPerWave);
  const int D = p.cfg.head_dim;
  if (p.cfg.act_dtype == C2KV_F32) {
    if (src_kind == SRC_PAGED) return launch_attn_d<float, SRC_PAGED>(D, ap, n, threads, st);
    return launch_attn_d<float, SRC_POOL>(D, ap, n, threads, st);
  }
  if (src_kind == SRC_PAGED) return launch_attn_d<__bf16, SRC_PAGED>(D, ap, n, threads, st);
  if (src_kind == SRC_POOL) return launch_attn_d<__bf16, SRC_POOL>(D, ap, n, threads, st);
  return launch_attn_d<__bf16, SRC_POOL_I8>(D, ap, n, threads, st);
}

hipError_t launch_merge(const Plan& p, void* out, float* lse, hipStream_t st) {
  if (p.merges.empty()) return hipSuccess;
  MergeParams mp{};
  mp.Hq = p.cfg.n_q_heads;
  mp.G = p.group;
  mp.S = p.suffix_len;
  mp.RB = p.rows_per_block;
  mp.groups = at<MergeGroup>(p.d_workspace, p.ws.merges);
  mp.part_o = at<float>(p.d_workspace, p.ws.part_o);
  mp.part_lse = at<float>(p.d_workspace, p.ws.part_lse);
  mp.out = out;
  mp.lse = lse;
  const int D = p.cfg.head_dim;
  const int rpw = 256 / (D / 4);
  const dim3 grid(static_cast<unsigned>(p.merges.size()), (p.rows_per_block + rpw - 1) / rpw);
  if (p.cfg.act_dtype == C2KV_F32) {
    if (D == 64) hipLaunchKernelGGL((merge_kernel<float, 64>), grid, dim3(256), 0, st, mp);
    else hipLaunchKernelGGL((merge_kernel<float, 128>), grid, dim3(256), 0, st, mp);
  } else {
    if (D == 64) hipLaunchKernelGGL((merge_kernel<__bf16, 64>), grid, dim3(256), 0, st, mp);
    else hipLaunchKernelGGL((merge_kernel<__bf16, 128>), grid, dim3(256), 0, st, mp);
  }
  return hipGetLastError();
}

hipError_t launch_compose(const Plan& p, int pool_dtype, const void* k, const void* v,
                          const float* k_scale, const float* v_scale, void* k_pages,
                          void* v_pages, int64_t* out_src_row, int32_t* out_pos,
                          hipStream_t st) {
  const int n_tiles = static_cast<int>(p.compose_tiles.size() / 2);
  if (n_tiles == 0) return hipSuccess;
  ComposeParams cp{};
  cp.Hkv = p.cfg.n_kv_heads;
  cp.PS = p.page_size;
  cp.max_pages = p.max_pages;
  cp.req_slot0 = at<int>(p.d_workspace, p.ws.req_slot0);
  cp.slot_src = at<int>(p.d_workspace, p.ws.slot_src);
  cp.slot_seg = at<int>(p.d_workspace, p.ws.slot_seg);
  cp.slot_pos = at<int>(p.d_workspace, p.ws.slot_pos);
  cp.seg_cs = at<float2>(p.d_workspace, p.ws.seg_cs);
  cp.block_table = at<int>(p.d_workspace, p.ws.block_table);
  cp.tiles = at<int>(p.d_workspace, p.ws.compose_tiles);
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
  if (p.cfg.act_dtype == C2KV_F32) {
    if (D == 64) hipLaunchKernelGGL((compose_kernel<float, 64, float>), grid, dim3(256), 0, st, cp);
    else hipLaunchKernelGGL((compose_kernel<float, 128, float>), grid, dim3(256), 0, st, cp);
  } else if (pool_dtype == C2KV_I8) {
    if (D == 64) hipLaunchKernelGGL((compose_kernel<__bf16, 64, int8_t>), grid, dim3(256), 0, st, cp);
    else hipLaunchKernelGGL((compose_kernel<__bf16, 128, int8_t>), grid, dim3(256), 0, st, cp);
  } else {
    if (D == 64) hipLaunchKernelGGL((compose_kernel<__bf16, 64, __bf16>), grid, dim3(256), 0, st, cp);
    else hipLaunchKernelGGL((compose_kernel<__bf16, 128, __bf16>), grid, dim3(256), 0, st, cp);
  }
  return hipGetLastError();
}

}  // namespace c2kv

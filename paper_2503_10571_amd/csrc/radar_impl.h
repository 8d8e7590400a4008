// Internal declarations shared by the translation units of libradar.so:
// the device helpers every kernel uses (sequence spans, element conversion,
// streaming loads, DPP exchanges, the top-k and union building blocks, the
// attention tile), the host-side shape and workspace types, the launch
// helper, and the launchers each unit provides to the others. Not part of
// the C ABI (include/radar.h is).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <type_traits>
#include <vector>

#include "radar.h"

namespace radar_impl {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr int kWave = 64;
constexpr int kTile = 64;          // tokens per wave in k_attend / k_build
constexpr int kMaxK = 256;         // largest k accepted
constexpr int kMaxG = 8;           // largest query-head group
constexpr int kMaxCand = 2048;     // largest number of candidate segments
constexpr int kMaxWg = 1024;       // largest attention split per (b, kv head)

typedef uint16_t bf16_t;           // storage type of a bfloat16 value
typedef unsigned long long u64;   // 64-bit type of the wave shuffles
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// token layout of one sequence at a decode step
// ---------------------------------------------------------------------------
// A sequence of length len starts with sink = min(n_sink, len) attention-sink
// tokens. The kernels address K / V from the first row after the sinks
// (the host offsets the pointers by n_sink rows), so in these row numbers
// candidate segment s covers [s c, s c + c) for s < n_cand, the window is
// [ws, t) with t = len - sink and ws = c floor(max(0, t - w) / c), and the
// sinks are rows [-n_sink, -n_sink + sink). A length outside [1, t_max]
// marks the sequence invalid: it selects nothing, attends nothing, and its
// outputs are NaN.
struct SeqArgs {
  const int64_t* lens;  // [B] per-sequence lengths (device), or null: all t_max
  int64_t t_max;
  int c, w, n_sink, k;
  int lens_add = 0;     // 1: lens holds append rows, a sequence's length is
                        // its row + 1 (0, invalid, unless row < t_max)
};

// Lengths stay below 2^31 (the capacity limit), so the split is computed in
// 32-bit arithmetic.
struct Span {
  int t, ws, n_cand, k_eff, sink;
  bool ok;
};

__host__ __device__ inline Span make_span(int64_t len, const SeqArgs& a) {
  Span p;
  p.ok = len >= 1 && len <= a.t_max;
  const int L = p.ok ? (int)len : 0;
  p.sink = L < a.n_sink ? L : a.n_sink;
  p.t = L - p.sink;
  const unsigned past = p.t > a.w ? (unsigned)(p.t - a.w) : 0u;
  p.n_cand = (int)(past / (unsigned)a.c);
  p.ws = p.n_cand * a.c;
  p.k_eff = p.n_cand < a.k ? p.n_cand : a.k;
  return p;
}

__device__ __forceinline__ Span seq_span(const SeqArgs& a, int64_t b) {
  if (!a.lens) return make_span(a.t_max, a);
  const int64_t v = a.lens[b];
  if (!a.lens_add) return make_span(v, a);
  return make_span(v >= 0 && v < a.t_max ? v + 1 : 0, a);
}

// The k / v row write of an append. radar_append runs it as its own kernel;
// radar_append_decode runs it inside the per-(b, kv head) kernel that
// precedes every read of the row, one wave per pair.
struct AppendArgs {
  uint4* K;                // cache base (row 0 of pair 0); null: no append
  uint4* V;
  const uint4* kn;         // [B][Hkv] rows of the new keys / values
  const uint4* vn;
  const int64_t* pos;      // [B] row of sequence b, or null: row t for all
  int64_t t;
  int chunks;              // 16-byte chunks per row
};

// rows outside [0, cap) are skipped
__device__ __forceinline__ void append_row(const AppendArgs& ap, int64_t cap,
                                           int64_t bh, int Hkv, int lane) {
  const int64_t row = ap.pos ? ap.pos[bh / Hkv] : ap.t;
  if (row < 0 || row >= cap) return;
  const int64_t dst = (bh * cap + row) * ap.chunks, src = bh * ap.chunks;
  for (int i = lane; i < ap.chunks; i += kWave) {
    ap.K[dst + i] = ap.kn[src + i];
    ap.V[dst + i] = ap.vn[src + i];
  }
}

// union entries: segment id in the low 16 bits, the mask of the group's
// query heads that selected it in bits 16 .. 23
constexpr int kUniIdBits = 16;
constexpr unsigned kAllHeads = 0xffu;

// ---------------------------------------------------------------------------
// element helpers
// ---------------------------------------------------------------------------
template <typename T> struct Elem;
template <> struct Elem<float> { static constexpr int kPer16 = 4; };
template <> struct Elem<bf16_t> { static constexpr int kPer16 = 8; };

__device__ __forceinline__ float bf16_lo(uint32_t x) {
  return __uint_as_float(x << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t x) {
  return __uint_as_float(x & 0xffff0000u);
}

// 16 bytes -> floats
template <typename T>
__device__ __forceinline__ void unpack16(const uint4& u, float* f);
template <>
__device__ __forceinline__ void unpack16<float>(const uint4& u, float* f) {
  f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
  f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
}
template <>
__device__ __forceinline__ void unpack16<bf16_t>(const uint4& u, float* f) {
  f[0] = bf16_lo(u.x); f[1] = bf16_hi(u.x);
  f[2] = bf16_lo(u.y); f[3] = bf16_hi(u.y);
  f[4] = bf16_lo(u.z); f[5] = bf16_hi(u.z);
  f[6] = bf16_lo(u.w); f[7] = bf16_hi(u.w);
}

// fp32 -> bf16, round to nearest even; infinities stay infinite and NaN
// becomes a quiet NaN (a select, not a branch)
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t qnan = (u >> 16) | 0x40u;
  return (u & 0x7fffffffu) > 0x7f800000u ? qnan : rounded;
}
__device__ __forceinline__ float round_bf16(float f) {
  return __uint_as_float(f32_to_bf16(f) << 16);
}

template <typename T> __device__ __forceinline__ T from_f32(float f);
template <> __device__ __forceinline__ float from_f32<float>(float f) { return f; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float f) {
  return (bf16_t)f32_to_bf16(f);
}
template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

// Non-temporal 16-byte loads for data read once per launch (K/V tiles, key
// tiles, summary rows): they stream past the caches and sustain a higher
// HBM read rate than ordinary loads on MI355X.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4v_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ float4 ld_stream_f4(const float* p) {
  const f32x4v_t t = __builtin_nontemporal_load(reinterpret_cast<const f32x4v_t*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}

// Omega is fp32 [n][d], or bf16 [n][d] for bf16 caches (whose projection
// rounds Omega to bf16 anyway, so both give the same products); four
// consecutive entries from element idx, widened to fp32 (exact for bf16).
// fp32 caches always pass fp32 Omega.
template <bool BF>
__device__ __forceinline__ float4 load_omega4(const void* omega, int64_t idx) {
  if constexpr (BF) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(omega) + idx);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(omega) + idx);
  }
}

// NR rows of QPL Omega entries (row_idx(p): element index of row p's first
// entry), stored as bf16 (BF) or fp32, all loads issued together and kept
// as raw words (fp32: four floats; bf16: four values in .x and .y);
// omega_f4 widens a word where it is used. Callers choose BF at compile
// time, so no branch or conversion sits between these loads and the loads
// issued after them.
template <bool BF, int NR, int QPL, typename F>
__device__ __forceinline__ void load_omega_rows(uint4 (&raw)[NR][QPL / 4], const void* omega,
                                                F&& row_idx) {
#pragma unroll
  for (int p = 0; p < NR; ++p)
#pragma unroll
    for (int e4 = 0; e4 < QPL / 4; ++e4) {
      if constexpr (BF) {
        const uint2 u = *reinterpret_cast<const uint2*>(
            static_cast<const uint16_t*>(omega) + row_idx(p) + 4 * e4);
        raw[p][e4] = make_uint4(u.x, u.y, 0u, 0u);
      } else {
        raw[p][e4] = *reinterpret_cast<const uint4*>(
            static_cast<const float*>(omega) + row_idx(p) + 4 * e4);
      }
    }
}
template <bool BF>
__device__ __forceinline__ float4 omega_f4(uint4 w) {
  if constexpr (BF)
    return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                       __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
  else
    return make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z),
                       __uint_as_float(w.w));
}

// ---------------------------------------------------------------------------
// cross-lane exchanges
// ---------------------------------------------------------------------------
// DPP controls (GFX9): quad_perm [1,0,3,2] and [2,3,0,1] swap neighbours at
// distance 1 and 2; row_half_mirror maps lane i of each 8-lane half-row to
// 7 - i, row_mirror maps lane i of each 16-lane row to 15 - i;
// row_newbcast:n copies lane n of every row to the whole row.
constexpr int kDppQuadSwap1 = 0xB1;
constexpr int kDppQuadSwap2 = 0x4E;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
constexpr int kDppRowBcast0 = 0x150;

// compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// (a plain DPP move, every lane's source valid for these controls: the
// compiler folds it into the add or max that consumes it)
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}

// Lanes l and l ^ 16 (MASK 16) or l and l ^ 32 (MASK 32) exchange on the
// vector ALUs: v_permlane16_swap / v_permlane32_swap with both operands the
// same value leave, in every lane, the pair's two values (the lower lane's
// first) in the two results.
template <int MASK>
__device__ __forceinline__ void xor_pair(float v, float& lo, float& hi) {
  static_assert(MASK == 16 || MASK == 32, "permlane swap distance");
  const unsigned u = __float_as_uint(v);
  if constexpr (MASK == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    lo = __uint_as_float(r[0]); hi = __uint_as_float(r[1]);
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    lo = __uint_as_float(r[0]); hi = __uint_as_float(r[1]);
  }
}
// v plus the value of lane l ^ MASK (MASK 16 or 32; the same sum in both
// lanes of the pair)
template <int MASK>
__device__ __forceinline__ float xor_sum(float v) {
  float lo, hi;
  xor_pair<MASK>(v, lo, hi);
  return lo + hi;
}

// Value of the partner lane in a pairing that differs from this lane in bit
// MASK. Within a 16-lane row the pairings are DPP moves (mirrors for bits 3
// and 2, quad swaps for bits 1 and 0); they are only used from the highest
// bit down, so the lower bits still to be processed never matter. Bits 4
// and 5 are lane l ^ MASK, by permlane swaps.
template <int MASK>
__device__ __forceinline__ float partner(float x, int lane) {
  if constexpr (MASK == 1) return dpp_f<kDppQuadSwap1>(x);
  else if constexpr (MASK == 2) return dpp_f<kDppQuadSwap2>(x);
  else if constexpr (MASK == 4) return dpp_f<kDppHalfMirror>(x);
  else if constexpr (MASK == 8) return dpp_f<kDppMirror>(x);
  else {
    float lo, hi;
    xor_pair<MASK>(x, lo, hi);
    return (lane & MASK) ? lo : hi;
  }
}

// One step of a cross-lane transpose-reduce: NV values per lane; paired lanes
// (different bit MASK) keep complementary halves, chosen by their own bit
// MASK, and add the partner's copy of the kept half.
template <int NV, int MASK>
__device__ __forceinline__ void halve(float* v, int lane) {
  const bool up = (lane & MASK) != 0;
#pragma unroll
  for (int i = 0; i < NV / 2; ++i) {
    const float keep = up ? v[i + NV / 2] : v[i];
    const float send = up ? v[i] : v[i + NV / 2];
    v[i] = keep + partner<MASK>(send, lane);
  }
}

// Reduce NV partial sums (one per row i) held by every lane of each group of
// NV consecutive lanes: afterwards lane j of the group holds row j's total.
template <int NV>
__device__ __forceinline__ void transpose_reduce(float* v, int lane) {
  if constexpr (NV >= 64) halve<64, 32>(v, lane);
  if constexpr (NV >= 32) halve<32, 16>(v, lane);
  if constexpr (NV >= 16) halve<16, 8>(v, lane);
  if constexpr (NV >= 8) halve<8, 4>(v, lane);
  if constexpr (NV >= 4) halve<4, 2>(v, lane);
  if constexpr (NV >= 2) halve<2, 1>(v, lane);
}

// 16-lane row all-reduce (every lane of a row ends with the row's result)
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, dpp_f<kDppQuadSwap1>(v));
  v = fmaxf(v, dpp_f<kDppQuadSwap2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  return fmaxf(v, dpp_f<kDppMirror>(v));
}
__device__ __forceinline__ float row_sum(float v) {
  v += dpp_f<kDppQuadSwap1>(v);
  v += dpp_f<kDppQuadSwap2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  return v + dpp_f<kDppMirror>(v);
}
__device__ __forceinline__ float lane_read(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
// wave-wide results, uniform across the wave (rows combined by readlane)
__device__ __forceinline__ float wave_max(float v) {
  v = row_max(v);
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)),
               fmaxf(lane_read(v, 32), lane_read(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = row_sum(v);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}


// ---------------------------------------------------------------------------
// top-k helpers
// ---------------------------------------------------------------------------
// Order key of (score, index): larger key = better; ties in score go to the
// lower segment index. Keys are unique because indices are; 0 = no segment.
__device__ __forceinline__ u64 order_key(float s, int idx) {
  uint32_t u = __float_as_uint(s);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((u64)u << 32) | (u64)(0xffffffffu - (uint32_t)idx);
}
__device__ __forceinline__ int key_index(u64 key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffu));
}
__device__ __forceinline__ float key_score(u64 key) {
  uint32_t u = (uint32_t)(key >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

// Top-k_eff of one query head by one wave, k-independent. Lane l holds
// candidates m * 64 + l (m < NPL: coalesced loads). The k_eff-th largest
// 32-bit score key is found bit by bit, from the highest bit in which the
// present keys differ down (the bits above it are common to all of them): at
// each bit every lane counts its keys that match the prefix found so far and
// have the bit set, a DPP reduction sums the counts, and the bit is kept
// when at least the still-needed number of keys has it. The search stops
// once every key matching the prefix is needed. Then every key above the
// threshold and the lowest-index keys equal to it are compacted into LDS
// (positions from a prefix sum of per-lane counts; only when more keys tie
// at the threshold than are needed does the index order of the ties take
// one ballot per register) and rank-sorted by (score desc, index asc).
// list: k words of LDS owned by this wave. Vector counts and scans: no LDS
// atomics (candidates of similar scores share their leading bits, so a
// histogram over those bits sends every key to one bin) and no ballot per
// key and bit.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, true);
}
// AND / OR over the 64 lanes, uniform: the 16-lane row by DPP (quad swaps,
// mirrors), then the rows by permlane swaps
__device__ __forceinline__ uint32_t wave_and_u32(uint32_t v) {
  int x = (int)v;
  x &= dpp_i<kDppQuadSwap1>(x);
  x &= dpp_i<kDppQuadSwap2>(x);
  x &= dpp_i<kDppHalfMirror>(x);
  x &= dpp_i<kDppMirror>(x);
  float lo, hi;
  xor_pair<16>(__int_as_float(x), lo, hi);
  x = __float_as_int(lo) & __float_as_int(hi);
  xor_pair<32>(__int_as_float(x), lo, hi);
  x = __float_as_int(lo) & __float_as_int(hi);
  return (uint32_t)__builtin_amdgcn_readfirstlane(x);
}
__device__ __forceinline__ uint32_t wave_or_u32(uint32_t v) {
  int x = (int)v;
  x |= dpp_i<kDppQuadSwap1>(x);
  x |= dpp_i<kDppQuadSwap2>(x);
  x |= dpp_i<kDppHalfMirror>(x);
  x |= dpp_i<kDppMirror>(x);
  float lo, hi;
  xor_pair<16>(__int_as_float(x), lo, hi);
  x = __float_as_int(lo) | __float_as_int(hi);
  xor_pair<32>(__int_as_float(x), lo, hi);
  x = __float_as_int(lo) | __float_as_int(hi);
  return (uint32_t)__builtin_amdgcn_readfirstlane(x);
}
// sum over the 64 lanes, uniform
__device__ __forceinline__ int wave_sum_i32(int v) {
  v += dpp_i<kDppQuadSwap1>(v);
  v += dpp_i<kDppQuadSwap2>(v);
  v += dpp_i<kDppHalfMirror>(v);
  v += dpp_i<kDppMirror>(v);
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}
// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
  int x = v;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15);
  const int r1 = __builtin_amdgcn_readlane(x, 31);
  const int r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = lane >> 4;
  return x + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}

template <int NPL>
__device__ void head_topk(const float* __restrict__ src, int n_cand, int k,
                          int k_eff, int* sel_row, int32_t* sel_out,
                          float* sc_out, int lane, u64* list) {
  uint32_t u[NPL];                         // ordered score keys, 0 = absent
  if (n_cand > 0) {
    float v[NPL];
#pragma unroll
    for (int m = 0; m < NPL; ++m) v[m] = src[min(m * 64 + lane, n_cand - 1)];
#pragma unroll
    for (int m = 0; m < NPL; ++m)
      u[m] = (m * 64 + lane < n_cand) ? (uint32_t)(order_key(v[m], 0) >> 32) : 0u;
  } else {
#pragma unroll
    for (int m = 0; m < NPL; ++m) u[m] = 0u;
  }
  if (k_eff > 0) {
    // bits common to every present key (absent keys count as neither)
    uint32_t kand = 0xffffffffu, kor = 0u;
#pragma unroll
    for (int m = 0; m < NPL; ++m)
      if (u[m] != 0u) { kand &= u[m]; kor |= u[m]; }
    kand = wave_and_u32(kand);
    kor = wave_or_u32(kor);
    const uint32_t diff = kand ^ kor;
    const int top = diff ? 31 - __clz((int)diff) : -1;
    // (prefix, mask): the leading bits of the k_eff-th largest key found so
    // far; `need` keys are still to take among those matching them (every
    // key with larger leading bits is taken)
    uint32_t mask = top >= 0 ? ~((2u << top) - 1u) : 0xffffffffu;
    uint32_t prefix = kand & mask;
    int need = k_eff;
#pragma unroll 1
    for (int bit = top; bit >= 0; --bit) {
      const uint32_t mb = mask | (1u << bit);
      const uint32_t pb = prefix | (1u << bit);
      int c = 0;
#pragma unroll
      for (int m = 0; m < NPL; ++m) c += ((u[m] & mb) == pb) ? 1 : 0;
      const int cnt = wave_sum_i32(c);
      mask = mb;
      if (cnt >= need) {
        prefix = pb;
        // every key left with these leading bits is taken
        if (cnt == need) break;
      } else {
        need -= cnt;
      }
    }
    // take every key whose leading bits are larger, and the `need`
    // lowest-index keys whose leading bits equal them
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
      const uint32_t um = u[m] & mask;
      n_gt += um > prefix ? 1 : 0;
      n_eq += (um == prefix && u[m] != 0u) ? 1 : 0;
    }
    const bool all_eq = wave_sum_i32(n_eq) == need;   // uniform
    // eq_take[m]: whether this lane's key m is a tie that is taken
    uint32_t eq_take = 0u;
    if (all_eq) {
#pragma unroll
      for (int m = 0; m < NPL; ++m)
        eq_take |= ((u[m] & mask) == prefix && u[m] != 0u) ? 1u << m : 0u;
    } else {
      // more ties than needed: the lowest indices, m * 64 + lane order
      const u64 lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      int before = 0;
#pragma unroll
      for (int m = 0; m < NPL; ++m) {
        const bool eq = (u[m] & mask) == prefix && u[m] != 0u;
        const u64 be = __ballot(eq);
        if (eq && before + (int)__popcll(be & lt_mask) < need) eq_take |= 1u << m;
        before += __popcll(be);
      }
    }
    const int n_take = n_gt + __popc(eq_take);
    int pos = wave_incl_scan(n_take, lane) - n_take;
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
      if ((u[m] & mask) > prefix || ((eq_take >> m) & 1u)) {
        list[pos] = ((u64)u[m] << 32) | (u64)(0xffffffffu - (uint32_t)(m * 64 + lane));
        ++pos;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // rank sort of the k_eff selected keys (larger key first)
    for (int i = lane; i < k_eff; i += 64) {
      const u64 key = list[i];
      int rank = 0;
#pragma unroll 8
      for (int j = 0; j < k_eff; ++j) rank += list[j] > key ? 1 : 0;
      const int idx = key_index(key);
      sel_row[rank] = idx;
      if (sel_out) sel_out[rank] = idx;
      if (sc_out) sc_out[rank] = key_score(key);
    }
  }
  for (int r = k_eff + lane; r < k; r += 64) {
    if (sel_out) sel_out[r] = -1;
    if (sc_out) sc_out[r] = __uint_as_float(0x7fc00000u);
  }
}

// Union of the group's selections: sel[h * per .. h * per + per) holds the
// segment ids of head h < G (-1 = none, every other id < kMaxCand). The ids
// are set in an LDS bitmap (one per head when masks are wanted); the first
// wave ORs the heads' words and turns the popcounts into prefix offsets, and
// then every thread of the workgroup lists some of the set bits: the
// distinct ids in ascending order go to uni, each with the mask of the heads
// that chose it (all heads without masks), and their count to *ucnt. bits:
// G * kMaxCand / 32 words of LDS. A barrier-synchronised call of the whole
// workgroup; the caller orders sel's writes before it and uni's reads after.
constexpr int kBitmapWords = kMaxCand / 32;
static_assert(kBitmapWords == kWave, "one bitmap word per lane");
__device__ inline void group_union(const int* sel, unsigned* bits, int G, int per,
                            bool masks, int* uni, int* ucnt) {
  // each word's union over the maps, and its exclusive prefix of set bits
  __shared__ uint32_t or_lds[kBitmapWords];
  __shared__ int pre_lds[kBitmapWords];
  const int tid = threadIdx.x;
  const int nmaps = masks ? G : 1;
  for (int i = tid; i < nmaps * kBitmapWords; i += blockDim.x) bits[i] = 0u;
  __syncthreads();
  for (int i = tid; i < G * per; i += blockDim.x) {
    const int id = sel[i];
    const int map = masks ? i / per : 0;
    if (id >= 0) atomicOr(&bits[map * kBitmapWords + (id >> 5)], 1u << (id & 31));
  }
  __syncthreads();
  if (tid < kWave) {
    uint32_t word = 0u;
    for (int g = 0; g < nmaps; ++g) word |= bits[g * kBitmapWords + tid];
    const int pc = __popc(word);
    // exclusive prefix sum of the popcounts over the 64 lanes
    int incl = pc;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int o = __shfl_up(incl, d);
      if (tid >= d) incl += o;
    }
    or_lds[tid] = word;
    pre_lds[tid] = incl - pc;
    if (tid == kWave - 1) *ucnt = incl;
  }
  __syncthreads();
  // every thread lists some of the set bits: id i sits at its word's
  // prefix plus the set bits below it in the word (ascending ids)
  for (int i = tid; i < kBitmapWords * 32; i += blockDim.x) {
    const int w = i >> 5, bit = i & 31;
    const uint32_t word = or_lds[w];
    if ((word >> bit) & 1u) {
      unsigned m = kAllHeads;
      if (masks) {
        m = 0u;
        for (int g = 0; g < nmaps; ++g) m |= ((bits[g * kBitmapWords + w] >> bit) & 1u) << g;
      }
      uni[pre_lds[w] + __popc(word & ((1u << bit) - 1u))] = i | (int)(m << kUniIdBits);
    }
  }
}

// ---------------------------------------------------------------------------
// exact attention over <= 64-token tiles (shared by k_attend and k_decode_fused)
// ---------------------------------------------------------------------------
// The attended tokens of a (b, kv head) are cut into tiles of <= 64 tokens
// that never cross a segment or the window boundary. A wave processes one
// tile at a time: lane (r, jj) (r = lane / LPR) reads the 16-byte chunk jj of
// rows r, r + RPI, ... so every load instruction covers RPI whole rows
// contiguously (rows past the tile end re-read its last row and are masked).
// q.k partials (bf16: v_dot2_f32_bf16 on the raw pairs, the scale applied to
// the sums; fp32: fma of the pre-scaled query) are transpose-reduced so that
// each lane ends with one token's logit, softmax runs across the wave, and p is broadcast back (DPP row
// broadcast) to the lanes that hold the matching V chunks. The state carries
// across tiles as an online softmax: running max m and sum l (log2 units,
// wave-uniform) and unreduced per-lane accumulators.
//
// (q.k on the matrix cores was measured slower here: the MFMA operand layout
// gives each 16-lane quarter of a load instruction one 16-byte chunk of 16
// different rows; that made one-head groups slower and groups of four no
// faster.)
template <typename T, int D, int G>
struct TileAttn {
  static constexpr int EPL = Elem<T>::kPer16;   // elements per 16-byte chunk
  static constexpr int LPR = D / EPL;           // lanes per row
  static constexpr int RPI = kWave / LPR;       // rows per load instruction
  static constexpr int ITER = kTile / RPI;      // load instructions per tile
  static_assert(ITER == LPR, "tile shape");

  // bf16: the raw query pairs (dot2 operands) and the scale applied to
  // the sums; fp32: the queries times the scale
  static constexpr bool BF = sizeof(T) == 2;
  float qf[BF ? 1 : G][EPL];
  uint32_t q2[BF ? G : 1][EPL / 2];
  float qs;
  float m[G], l[G], acc[G][EPL];

  // q0: the group's first query head; qscale folds log2(e) / sqrt(d)
  __device__ __forceinline__ void init(const T* __restrict__ q0, float qscale,
                                       int lane) {
    const int jj = lane % LPR;
    qs = qscale;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint4 u = *reinterpret_cast<const uint4*>(q0 + g * D + jj * EPL);
      if constexpr (BF) {
        q2[g][0] = u.x; q2[g][1] = u.y; q2[g][2] = u.z; q2[g][3] = u.w;
      } else {
        unpack16<T>(u, qf[g]);
#pragma unroll
        for (int e = 0; e < EPL; ++e) qf[g][e] *= qscale;
      }
      m[g] = -INFINITY;
      l[g] = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
    }
  }

  // rows [row0, row0 + len) of K and V (row0 counts rows from the base
  // pointers); 1 <= len <= 64; wave-uniform call. Head g of the group takes
  // part only if bit g of hmask is set (a head that has attended nothing
  // yet keeps m = -inf, l = 0, acc = 0).
  __device__ __forceinline__ void tile(const T* __restrict__ K,
                                       const T* __restrict__ V, int64_t row0,
                                       int len, int lane, unsigned hmask) {
    const int r = lane / LPR;
    const int jj = lane % LPR;
    uint4 kr[ITER], vr[ITER];
    if (BF && len == kTile) {              // uniform: no row to clamp
      const T* kbase = K + (row0 + r) * D + jj * EPL;
      const T* vbase = V + (row0 + r) * D + jj * EPL;
#pragma unroll
      for (int i = 0; i < ITER; ++i) kr[i] = ld_stream(kbase + i * RPI * D);
#pragma unroll
      for (int i = 0; i < ITER; ++i) vr[i] = ld_stream(vbase + i * RPI * D);
    } else {
      const T* kbase = K + row0 * D + jj * EPL;
      const T* vbase = V + row0 * D + jj * EPL;
#pragma unroll
      for (int i = 0; i < ITER; ++i)
        kr[i] = ld_stream(kbase + (int64_t)min(i * RPI + r, len - 1) * D);
#pragma unroll
      for (int i = 0; i < ITER; ++i)
        vr[i] = ld_stream(vbase + (int64_t)min(i * RPI + r, len - 1) * D);
    }

    // logits: lane (r, jj) ends with the logit of tile row jj * RPI + r
    float lg[G];
    {
      float pl[G][ITER];
#pragma unroll
      for (int i = 0; i < ITER; ++i) {
        if constexpr (BF) {
          // bf16 pairs: exact products, fp32 sums
          const uint32_t kw[4] = {kr[i].x, kr[i].y, kr[i].z, kr[i].w};
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float a = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w)
              a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v_t, q2[g][w]),
                                                  __builtin_bit_cast(bf16x2v_t, kw[w]), a,
                                                  false);
            pl[g][i] = a;
          }
        } else {
          float kf[EPL];
          unpack16<T>(kr[i], kf);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float a = 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) a = fmaf(qf[g][e], kf[e], a);
            pl[g][i] = a;
          }
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        transpose_reduce<LPR>(pl[g], lane);
        lg[g] = BF ? pl[g][0] * qs : pl[g][0];
      }
    }
    const bool mine_ok = (jj * RPI + r) < len;
    float p[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const bool on = mine_ok && ((hmask >> g) & 1u);
      const float mt = wave_max(on ? lg[g] : -INFINITY);
      const float mn = fmaxf(m[g], mt);
      const float mref = mn == -INFINITY ? 0.f : mn;
      const float scale = fast_exp2(m[g] - mref);  // 0 on the head's first tile
      p[g] = on ? fast_exp2(lg[g] - mref) : 0.f;
      l[g] = fmaf(l[g], scale, wave_sum(p[g]));
      m[g] = mn;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] *= scale;
    }
    static_for<0, ITER>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      float vf[EPL];
      unpack16<T>(vr[i], vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        // p of row (i, r) lives in lane i of this lane's LPR-lane group
        float pb;
        if constexpr (LPR == 16)
          pb = dpp_f<kDppRowBcast0 + i>(p[g]);
        else
          pb = __shfl(p[g], r * LPR + i);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(pb, vf[e], acc[g][e]);
      }
    });
  }

  // sum the accumulators over the RPI row groups: lanes r = 0 (lane < LPR)
  // then hold dims jj*EPL .. jj*EPL + EPL - 1 of the wave's total
  __device__ __forceinline__ void reduce_rows() {
    static_for<0, 6>([&](auto bc) {
      constexpr int msk = 1 << decltype(bc)::value;
      if constexpr (msk >= LPR) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int e = 0; e < EPL; ++e) {
            if constexpr (msk >= 16) acc[g][e] = xor_sum<msk>(acc[g][e]);
            else acc[g][e] += __shfl_xor(acc[g][e], msk);
          }
      }
    });
  }
};

// decode path shared by the fused kernel and its select-only instantiation
// k_decode_fused modes: the whole step; the selection only (select path);
// the step from scores the split path's kernels computed (scored path)
constexpr int kFusedFull = 0;
constexpr int kFusedSelect = 1;
constexpr int kFusedScored = 2;
constexpr int kFusedWaves = 8;
constexpr int kFusedMaxG = 4;
constexpr int kFusedMaxCand = 1024;

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
// text of the last HIP error seen by this thread
extern thread_local char g_last_error[256];
// phase-clock buffer of the fused kernel's launches from this thread (null:
// off) and the number of workgroups it has room for
extern thread_local uint64_t* g_clock;
extern thread_local int g_clock_max;

// ---- launch helper with optional per-kernel event timing -----------------
// While profiling is enabled on a host thread, every launch goes through
// hipExtLaunchKernelGGL with a start/stop event pair, so the recorded times
// bracket exactly that kernel's execution on its stream.
// Read records return their events to a pool, so a profiled pass that
// follows another creates no events (event creation is host work that would
// otherwise slow the launches being timed).
struct Profiler {
  bool on = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  bool take(hipEvent_t* e) {
    if (!pool.empty()) { *e = pool.back(); pool.pop_back(); return true; }
    return hipEventCreate(e) == hipSuccess;
  }
};
extern thread_local Profiler g_prof;

template <typename F, typename... Args>
inline void launch(int kind, F kern, dim3 grid, dim3 block, size_t shm, hipStream_t st,
            Args... args) {
  if (g_prof.on) {
    hipEvent_t a = nullptr, b = nullptr;
    if (g_prof.take(&a)) {
      if (g_prof.take(&b)) {
        hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)shm, st, a, b, 0u, args...);
        g_prof.recs.push_back({kind, a, b});
        return;
      }
      g_prof.pool.push_back(a);
    }
  }
  hipLaunchKernelGGL(kern, grid, block, shm, st, args...);
}

struct Shape {
  int B, Hq, Hkv, G, d, n, c, w, n_sink, per_head;
  int64_t cap, s_cap;
  radar_dtype dt;
  bool obf;                                // Omega stored as bf16
};

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct WsLayout {
  size_t phiq, scores, uni, ucnt, part, total;
  int umax, maxwg, tiles_per_seg;
};

// RADAR_EHIP with the HIP error text recorded, or RADAR_OK
radar_status launch_status();

// compute units of the current device
int num_cu();

// K / V rows after the n_sink sink rows of the first (b, kv head): the
// kernels address segments and the window from there
// K / V rows after the n_sink sink rows of the first (b, kv head): the
// kernels address segments and the window from there
template <typename P>
P* after_sinks(const Shape& s, P* p) {
  const size_t esz = s.dt == RADAR_BF16 ? 2 : 4;
  using B = typename std::conditional<std::is_const<P>::value, const unsigned char,
                                      unsigned char>::type;
  return reinterpret_cast<P*>(reinterpret_cast<B*>(p) + (size_t)s.n_sink * s.d * esz);
}

// Split of the attention work (see attend_grid).
struct AttendGrid {
  int grid_x, tpw;
};

// ---- launchers provided by the units ---------------------------------------
// build.hip: segment summaries of segments [seg_first, seg_first + seg_count)
// of every (b, kv head), or with pos the per-sequence segment closes; K
// starts after the sinks
radar_status launch_build(const Shape& s, const void* K, const void* omega,
                          float* summ, int seg_first, int seg_count,
                          const int64_t* pos, hipStream_t st);

// split.hip: the split path's stages
void launch_phi_q_any(const Shape& s, const void* q, const void* omega, float* phiq,
                      hipStream_t st);
void launch_score(const Shape& s, const float* phiq, const float* summ,
                  float* scores, int n_cand, const SeqArgs& sa, hipStream_t st);
// ln(beta) of candidates [0, n_cand) into rows of nc_cap scores; with_rest
// also the mass of the window and sinks at index n_cand
void launch_segment_mass(const Shape& s, const void* q, const void* K, float* scores,
                         int n_cand, const SeqArgs& sa, int nc_cap, bool with_rest,
                         hipStream_t st);
void launch_topk_union(const Shape& s, const float* scores, const SeqArgs& sa,
                       int* uni, int* ucnt, int umax, int32_t* selected,
                       float* sel_scores, const AppendArgs& ap, hipStream_t st);
void launch_union_given(const Shape& s, const int32_t* given, int given_k,
                        const SeqArgs& sa, int* uni, int* ucnt, int umax,
                        hipStream_t st);
int64_t extra_tiles(const Shape& s, const SeqArgs& sa);
AttendGrid attend_grid(const Shape& s, const WsLayout& L, int u_bound, int64_t extra);
radar_status launch_attend(const Shape& s, const void* q, const void* K,
                           const void* V, const AttendGrid& ag, const SeqArgs& sa,
                           void* out, unsigned char* w, const WsLayout& L,
                           hipStream_t st);
void launch_combine_any(const Shape& s, const float* part, const int* ucnt, void* out,
                        const SeqArgs& sa, const WsLayout& L, int tpw, int fixed_nwg,
                        int partials_per_head, hipStream_t st);

// fused.hip (one unit per feature count n): the fused decode kernel, or with
// sel its select-only instantiation that hands the union to the split path
struct FusedArgs {
  const Shape* s;
  const void *q, *K, *V, *omega;
  const float* summ;
  SeqArgs sa;
  void* out;
  int32_t* selected;
  float* sel_scores;
  int *uni_out, *ucnt_out;
  int umax;
  AppendArgs ap;
  int R;
  float* part;
  int maxwg;
  hipStream_t st;
  const float* gscores;    // scored path: [B][Hq][nc_cap] Eq. 6 scores
  int nc_cap;
};
radar_status launch_fused_n64(const FusedArgs& a, bool sel);
radar_status launch_fused_n128(const FusedArgs& a, bool sel);
radar_status launch_fused_n256(const FusedArgs& a, bool sel);
radar_status launch_fused_n512(const FusedArgs& a, bool sel);
radar_status launch_fused_n1024(const FusedArgs& a, bool sel);
radar_status launch_fused_n2048(const FusedArgs& a, bool sel);
// (fused_n64 unit) the fused kernel from phase 3 on, over gscores
radar_status launch_fused_scored(const FusedArgs& a);

}  // namespace radar_impl

// Radar decode path on MI355X (gfx950, CDNA4): kernels and the C ABI.
//
// Kernels (all on the caller's stream):
//   k_build        segment summaries, Eq. 4 + Eq. 5: bf16/fp32 matrix-core
//                  projection of the keys onto Omega, exp2 epilogue, mean
//                  over the segment's tokens. Also serves the segment close
//                  of an append, so appends and rebuilds agree bit for bit.
//   k_append       writes one k/v row per (b, kv head) (radar_append; in
//                  radar_append_decode the decode's first per-pair kernel
//                  writes the rows instead).
//   k_decode_fused the whole decode step of one (b, kv head) in one
//                  workgroup: phi(q), Eq. 6 scores, top-k, union, attention
//                  and merge. Its select-only instantiation (phases up to the
//                  union) is the first kernel of the select path.
//   k_phi_q        phi(q), Eq. 4, per block of 64 features of a kv head's
//                  query group (split path).
//   k_score        Eq. 6 scores of every candidate segment: HBM-bound GEMV
//                  over the fp32 summaries, DPP transpose-reduce.
//   k_topk_union   per query head top-k (score desc, index asc) by radix
//                  selection; per kv head sorted union of the group.
//   k_segment_mass ln(beta_s), the exact attention mass of every candidate
//                  segment (the exact-selection ablation).
//   k_union_given  union of caller-given selections.
//   k_attend       exact attention (Eq. 1-2) over the union's segments plus
//                  the window and sinks: coalesced 16-byte gathers of K/V,
//                  fp32 online softmax, one partial (max, sum, acc[d]) per
//                  workgroup.
//   k_combine      log-sum-exp merge of the partials into the output.
//   k_peak_mfma, k_peak_exp  measurement microkernels (matrix and exp2 rates).
//
// Stages hand data to each other only inside a workgroup (LDS) or across
// kernel boundaries: the eight L2 caches of the chip are not coherent with
// one another, and the fences a cross-workgroup hand-off would need flush
// them.
//
// All softmax / feature exponentials are base 2 with log2(e) folded into the
// scale factors: exp(x) = exp2(x * log2(e)).

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <type_traits>
#include <vector>

#include "radar.h"

namespace {

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

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(
      __float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// Value of the partner lane in a pairing that differs from this lane in bit
// MASK. Within a 16-lane row the pairings are DPP moves (mirrors for bits 3
// and 2, quad swaps for bits 1 and 0); they are only used from the highest
// bit down, so the lower bits still to be processed never matter.
template <int MASK>
__device__ __forceinline__ float partner(float x) {
  if constexpr (MASK == 1) return dpp_f<kDppQuadSwap1>(x);
  else if constexpr (MASK == 2) return dpp_f<kDppQuadSwap2>(x);
  else if constexpr (MASK == 4) return dpp_f<kDppHalfMirror>(x);
  else if constexpr (MASK == 8) return dpp_f<kDppMirror>(x);
  else return __shfl_xor(x, MASK);
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
    v[i] = keep + partner<MASK>(send);
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
// k_build: segment summaries (Eq. 4, Eq. 5)
// ---------------------------------------------------------------------------
// Work item = one (b, kv head, segment) and one slice of 64*FT features.
// Wave w of the workgroup owns features [w*16*FT, (w+1)*16*FT) of the slice
// and keeps that slice of Omega (rounded to the MFMA input type) resident in
// registers as MFMA B operands for the whole kernel. Keys stream through two
// LDS buffers in tiles of 64 tokens (register-prefetched one tile ahead, one
// barrier per tile); every wave
// multiplies each 16-token sub-tile with its Omega slice on the matrix cores,
// applies exp2(acc * s1 - |k|^2 * s2) and adds the result into per-lane
// column sums. At the segment's end the sums are reduced across the four
// row groups of the MFMA output and scaled by 1 / (c sqrt(n)).
//
// MFMA operand layout (16x16 output tiles, both instructions):
//   A (keys):    lane l supplies row (l & 15), k-slots of group (l >> 4)
//   B (Omega^T): lane l supplies column (l & 15), same k-slots
//   D:           lane l holds rows 4*(l >> 4) + j, j < 4, column (l & 15)
// The k-slot -> head-dim map is the same for A and B, so the dot products
// are the same whatever order the hardware sums them in.
template <typename T> struct MfmaCfg;
template <> struct MfmaCfg<bf16_t> {     // v_mfma_f32_16x16x32_bf16
  static constexpr int kK = 32;          // head dims per instruction
  typedef bf16x8_t frag_t;
};
template <> struct MfmaCfg<float> {      // v_mfma_f32_16x16x4_f32
  static constexpr int kK = 4;
  typedef float frag_t;
};

template <typename T, int D>
struct BuildTile {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kPitch = kRowBytes + 16;          // LDS row pitch
  static constexpr int kChunksPerRow = kRowBytes / 16;
  static constexpr int kChunksPerThread = kTile * kChunksPerRow / 256;
};

template <typename T, int D, int FT>
__global__ __launch_bounds__(256) void k_build(
    const T* __restrict__ K, const void* __restrict__ omega, bool obf,
    float* __restrict__ summ, int n, int c, int64_t cap, int64_t s_cap,
    int seg_first, int seg_count, int64_t n_items, float s1, float s2,
    float out_scale, int64_t kv_head_stride_rows,
    const int64_t* __restrict__ pos, int Hkv, int n_sink) {
  using MC = MfmaCfg<T>;
  using BT = BuildTile<T, D>;
  constexpr int KB = D / MC::kK;
  constexpr int CPR = BT::kChunksPerRow;
  constexpr int CPT = BT::kChunksPerThread;
  static_assert(CPT >= 1 && (256 % CPR) == 0, "tile shape");

  __shared__ __attribute__((aligned(16))) unsigned char tile_lds[2][kTile * BT::kPitch];
  __shared__ float nrm_lds[2][kTile];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int fbase = blockIdx.y * (64 * FT) + wave * (16 * FT);

  // Omega slice -> B fragments (resident for the whole kernel)
  typename MC::frag_t bfrag[FT][KB];
#pragma unroll
  for (int f = 0; f < FT; ++f) {
    const int64_t orow = (int64_t)(fbase + f * 16 + col) * D;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if constexpr (sizeof(T) == 2) {
        const int64_t i0 = orow + kb * 32 + grp * 8;
        const float4 a = obf ? load_omega4<true>(omega, i0) : load_omega4<false>(omega, i0);
        const float4 b = obf ? load_omega4<true>(omega, i0 + 4) : load_omega4<false>(omega, i0 + 4);
        bf16x8_t v;
        v[0] = (short)f32_to_bf16(a.x); v[1] = (short)f32_to_bf16(a.y);
        v[2] = (short)f32_to_bf16(a.z); v[3] = (short)f32_to_bf16(a.w);
        v[4] = (short)f32_to_bf16(b.x); v[5] = (short)f32_to_bf16(b.y);
        v[6] = (short)f32_to_bf16(b.z); v[7] = (short)f32_to_bf16(b.w);
        bfrag[f][kb] = v;
      } else {
        bfrag[f][kb] = static_cast<const float*>(omega)[orow + kb * 4 + grp];
      }
    }
  }

  const int ntiles = (c + kTile - 1) / kTile;
  float psum[FT];
#pragma unroll
  for (int f = 0; f < FT; ++f) psum[f] = 0.f;

  // Segment of an item (one (b, kv head, segment); 32-bit arithmetic, item
  // counts stay below 2^31): seg_first + item % seg_count, or, with pos
  // (item = (b, kv head), one per-sequence segment close), the segment that
  // row pos[b] completes, -1 if it completes none. Rows count from the
  // first row after the n_sink sinks, where the K pointer starts.
  auto seg_of = [&](int64_t it) -> int {
    const uint32_t u = (uint32_t)it;
    if (!pos) return seg_first + (int)(u % (uint32_t)seg_count);
    const int64_t p = pos[u / (uint32_t)Hkv];
    const int64_t r = p - n_sink;
    if (p >= cap || r < 0 || (r + 1) % c != 0) return -1;
    return (int)((r + 1) / c - 1);
  };
  // first active item at or after it on this workgroup's stride
  auto next_active = [&](int64_t it) -> int64_t {
    while (it < n_items && seg_of(it) < 0) it += gridDim.x;
    return it;
  };
  // base row pointer of an item, computed once per segment
  auto item_base = [&](int64_t it) -> const T* {
    const uint32_t bh = (uint32_t)it / (uint32_t)seg_count;
    return K + ((int64_t)bh * kv_head_stride_rows + (int64_t)seg_of(it) * c) * D;
  };

  uint4 pre[CPT];
  int pre_valid = 0;
  // tile tl of the item whose rows start at `base`
  auto fetch = [&](const T* base, int tl_) {
    pre_valid = min(kTile, c - tl_ * kTile);
    const T* src = base + (int64_t)tl_ * kTile * D;
#pragma unroll
    for (int p = 0; p < CPT; ++p) {
      const int ci = p * 256 + tid;
      // rows past the segment re-read its last row; they are masked out
      // of the sums below
      const int row = min(ci / CPR, pre_valid - 1), ch = ci % CPR;
      pre[p] = ld_stream(reinterpret_cast<const unsigned char*>(src + (int64_t)row * D) +
                         ch * 16);
    }
  };
  // registers -> LDS buffer `buf`, with |k|^2 * s2 per row: the CPR chunks
  // of a row sit in CPR consecutive lanes, summed by DPP row reductions
  auto stage = [&](int buf) {
    unsigned char* tb = tile_lds[buf];
#pragma unroll
    for (int p = 0; p < CPT; ++p) {
      const int ci = p * 256 + tid;
      const int row = ci / CPR, ch = ci % CPR;
      *reinterpret_cast<uint4*>(tb + row * BT::kPitch + ch * 16) = pre[p];
      float sq = 0.f;
      if constexpr (sizeof(T) == 2) {
        // bf16 pairs: one dot2 per 32-bit word (exact products, fp32 sum)
        const uint32_t w[4] = {pre[p].x, pre[p].y, pre[p].z, pre[p].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bf16x2v_t v = __builtin_bit_cast(bf16x2v_t, w[i]);
          sq = __builtin_amdgcn_fdot2_f32_bf16(v, v, sq, false);
        }
      } else {
        float e[4];
        unpack16<T>(pre[p], e);
#pragma unroll
        for (int i = 0; i < 4; ++i) sq = fmaf(e[i], e[i], sq);
      }
      if constexpr (CPR == 8) {
        sq += dpp_f<kDppQuadSwap1>(sq);
        sq += dpp_f<kDppQuadSwap2>(sq);
        sq += dpp_f<kDppHalfMirror>(sq);
      } else {
        sq = row_sum(sq);
        if constexpr (CPR == 32) sq += __shfl_xor(sq, 16);
      }
      if (ch == 0) nrm_lds[buf][row] = sq * s2;
    }
  };

  // 16-token sub-tiles of the tile in `buf`; FULL: no rows to mask
  auto compute = [&](int buf, int valid, auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    const unsigned char* tb = tile_lds[buf];
#pragma unroll
    for (int st = 0; st < kTile / 16; ++st) {
      if (!FULL && st * 16 >= valid) break;
      typename MC::frag_t afrag[KB];
      const unsigned char* arow = tb + (st * 16 + col) * BT::kPitch;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        if constexpr (sizeof(T) == 2)
          afrag[kb] = *reinterpret_cast<const bf16x8_t*>(arow + (kb * 32 + grp * 8) * 2);
        else
          afrag[kb] = *reinterpret_cast<const float*>(arow + (kb * 4 + grp) * 4);
      }
      float nb[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) nb[j] = nrm_lds[buf][st * 16 + grp * 4 + j];
      // head-dim block outer, feature tile inner: FT independent
      // accumulation chains keep the matrix pipe busy
      f32x4_t acc[FT];
#pragma unroll
      for (int f = 0; f < FT; ++f) acc[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int f = 0; f < FT; ++f) {
          if constexpr (sizeof(T) == 2)
            acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[kb], bfrag[f][kb], acc[f], 0, 0, 0);
          else
            acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(afrag[kb], bfrag[f][kb], acc[f], 0, 0, 0);
        }
#pragma unroll
      for (int f = 0; f < FT; ++f)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float v = fast_exp2(fmaf(acc[f][j], s1, -nb[j]));
          if (FULL) psum[f] += v;
          else psum[f] += (st * 16 + grp * 4 + j < valid) ? v : 0.f;
        }
    }
  };

  // Pipeline, one barrier per tile: tile i is multiplied from one LDS buffer
  // while tile i+1 is in flight to registers; after the multiply the
  // registers go to the other buffer.
  int64_t item = next_active(blockIdx.x);
  int tl = 0, buf = 0;
  const T* base = nullptr;
  if (item < n_items) {
    base = item_base(item);
    fetch(base, 0);
    stage(0);
  }
  int valid = pre_valid;
  __syncthreads();
  while (item < n_items) {
    int64_t nitem = item;
    int ntl = tl + 1;
    const T* nbase = base;
    if (ntl == ntiles) {
      nitem = next_active(nitem + gridDim.x);
      ntl = 0;
      if (nitem < n_items) nbase = item_base(nitem);
    }
    const bool more = nitem < n_items;
    if (more) fetch(nbase, ntl);

    if (valid == kTile) compute(buf, valid, std::true_type{});
    else compute(buf, valid, std::false_type{});

    if (tl == ntiles - 1) {                // segment complete
      const int64_t bh = (uint32_t)item / (uint32_t)seg_count;
      const int64_t sg = seg_of(item);
      float* dst = summ + (bh * s_cap + sg) * n + fbase;
#pragma unroll
      for (int f = 0; f < FT; ++f) {
        float v = psum[f];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (lane < 16) dst[f * 16 + col] = v * out_scale;
        psum[f] = 0.f;
      }
    }
    if (more) stage(buf ^ 1);
    __syncthreads();
    buf ^= 1;
    valid = pre_valid;
    item = nitem;
    tl = ntl;
    base = nbase;
  }
}

// ---------------------------------------------------------------------------
// measurement microkernels (not part of the method)
// ---------------------------------------------------------------------------
// The two resources the index build spends: dense bf16 matrix-core work
// (8 independent 16x16x32 accumulation chains per wave) and exp2 on the
// vector ALUs (8 independent chains per lane). The sink store, which the
// compiler cannot prove dead, keeps the work alive.
constexpr int kPeakWgPerCu = 2;

__global__ __launch_bounds__(256) void k_peak_mfma(int iters, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (short)(0x3f80 + ((lane + i) & 7));     // bf16 values near 1
    b[i] = (short)(0x3f80 - i);
  }
  f32x4_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
  }
  float v = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) v += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = v;
}

__global__ __launch_bounds__(256) void k_peak_exp(int iters, float* __restrict__ sink) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = 1e-3f * (float)(threadIdx.x & 63) + 1e-2f * (float)j;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = fast_exp2(-x[j]);
  }
  float v = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) v += x[j];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = v;
}

// ---------------------------------------------------------------------------
// k_append: K[b][h][t] = k_new[b][h], V likewise (row pos[b] of sequence b
// when pos is given); one wave per (b, kv head)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_append(AppendArgs ap, int64_t cap, int Hkv) {
  append_row(ap, cap, blockIdx.x, Hkv, threadIdx.x);
}

// ---------------------------------------------------------------------------
// k_phi_q: phi(q) (Eq. 4) of the G query heads of one (b, kv head), one
// block of 64 features per workgroup
// ---------------------------------------------------------------------------
// Grid (n / 64, B * Hkv): each workgroup reads only its 64 rows of Omega.
// 16 lanes share one Omega row (D/16 floats each); wave w covers rows
// 16 w .. 16 w + 15 in 4 passes of 4 rows, and the 4 partial sums of each
// lane are reduced across its 16 lanes (transpose-reduce over 4 lanes, then
// two butterflies), so lane jj < 4 of row group r ends with feature
// 16 w + 4 jj + r.
template <typename T, int D, int G, bool BF>
__global__ __launch_bounds__(256) void k_phi_q(const T* __restrict__ q,
                                               const void* __restrict__ omega,
                                               float* __restrict__ phiq,
                                               int n, int Hq, int Hkv, float s1,
                                               float s2, float inv_sqrt_n) {
  constexpr int QPL = D / 16;              // q elements per lane
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane >> 4, jj = lane & 15;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int64_t hq0 = b * Hq + hk * G;     // the group's first (b, q head)
  const int f0 = blockIdx.x * 64 + wave * 16;

  uint4 om[4][QPL / 4];
  load_omega_rows<BF, 4, QPL>(om, omega, [&](int p) {
    return (int64_t)(f0 + p * 4 + r) * D + jj * QPL;
  });
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float qv[QPL];
#pragma unroll
    for (int e = 0; e < QPL; ++e) qv[e] = to_f32<T>(q[(hq0 + g) * D + jj * QPL + e]);
    float nrm = 0.f;
#pragma unroll
    for (int e = 0; e < QPL; ++e) nrm = fmaf(qv[e], qv[e], nrm);
    nrm = row_sum(nrm);
    float part[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      float a = 0.f;
#pragma unroll
      for (int e4 = 0; e4 < QPL / 4; ++e4) {
        float4 o = omega_f4<BF>(om[p][e4]);
        if constexpr (sizeof(T) == 2 && !BF) {
          o.x = round_bf16(o.x); o.y = round_bf16(o.y);
          o.z = round_bf16(o.z); o.w = round_bf16(o.w);
        }
        a = fmaf(o.x, qv[4 * e4], a);
        a = fmaf(o.y, qv[4 * e4 + 1], a);
        a = fmaf(o.z, qv[4 * e4 + 2], a);
        a = fmaf(o.w, qv[4 * e4 + 3], a);
      }
      part[p] = a;
    }
    transpose_reduce<4>(part, lane);
    float v = part[0];
    v += __shfl_xor(v, 4);
    v += __shfl_xor(v, 8);
    if (jj < 4)
      phiq[(hq0 + g) * n + f0 + jj * 4 + r] =
          fast_exp2(fmaf(v, s1, -nrm * s2)) * inv_sqrt_n;
  }
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

// Top-k_eff of one query head by one wave, k-independent: radix selection of
// the k_eff-th largest 32-bit score key in up to four 8-bit passes (a
// 256-bin LDS histogram of the keys that still match the prefix found so
// far, a suffix count over the bins by DPP row scans and readlanes, and a
// ballot for the bin holding the k_eff-th key; the passes stop early once
// every key left in that bin is needed), then a ballot rank among keys equal
// to that threshold (lower segment index first), compaction of the k_eff
// selected keys into LDS and a rank sort by (score desc, index asc).
// hist: 256 words and list: k words of LDS owned by this wave.
__device__ __forceinline__ int row_incl_scan(int v, int lane) {
  // inclusive prefix sum over the 64 lanes
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
                          float* sc_out, int lane, unsigned* hist, u64* list) {
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
    uint32_t prefix = 0u, mask = 0u;
    int need = k_eff;                      // keys still to take at or below prefix
#pragma unroll 1
    for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) hist[lane * 4 + i] = 0u;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int m = 0; m < NPL; ++m)
        if (u[m] != 0u && (u[m] & mask) == prefix)
          atomicAdd(&hist[(u[m] >> shift) & 255u], 1u);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // lane l owns bins 255 - 4l - j (j = 0..3): lane order runs from the
      // largest digit down, so a prefix over lanes counts larger digits
      int c[4], tot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) { c[j] = (int)hist[255 - lane * 4 - j]; tot += c[j]; }
      const int above = row_incl_scan(tot, lane) - tot;   // keys in larger digits
      int cum = above, pick = -1, before = 0, in_bin = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (pick < 0 && cum < need && need <= cum + c[j]) {
          pick = j; before = cum; in_bin = c[j];
        }
        cum += c[j];
      }
      const u64 who = __ballot(pick >= 0);
      const int wl = __ffsll((unsigned long long)who) - 1;
      const int pj = __builtin_amdgcn_readlane(pick, wl);
      const int pb = __builtin_amdgcn_readlane(before, wl);
      const int pc = __builtin_amdgcn_readlane(in_bin, wl);
      const uint32_t digit = 255u - (uint32_t)(wl * 4 + pj);
      prefix |= digit << shift;
      mask |= 255u << shift;
      need -= pb;
      // every key left in the chosen bin is taken: the digits found so far
      // already separate the k_eff largest keys from the rest
      if (need == pc) break;
    }
    // (prefix, mask) hold the leading digits of the k_eff-th largest key;
    // take every key whose leading digits are larger, and the `need`
    // lowest-index keys whose leading digits equal them (all of them when
    // the passes stopped early)
    int eq_before = 0;
    int n_sel = 0;
    const u64 lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
      const uint32_t um = u[m] & mask;
      const bool eq = um == prefix && u[m] != 0u;
      const u64 be = __ballot(eq);
      const bool take = (um > prefix) ||
                        (eq && eq_before + (int)__popcll(be & lt_mask) < need);
      eq_before += __popcll(be);
      const u64 bt = __ballot(take);
      if (take) {
        const int pos = n_sel + __popcll(bt & lt_mask);
        const int idx = m * 64 + lane;
        list[pos] = ((u64)u[m] << 32) | (u64)(0xffffffffu - (uint32_t)idx);
      }
      n_sel += __popcll(bt);
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
// wave ORs the heads' words, turns the popcounts into prefix offsets, and
// each lane lists its word's set bits: the distinct ids in ascending order go
// to uni, each with the mask of the heads that chose it (all heads without
// masks), and their count to *ucnt. bits: G * kMaxCand / 32 words of LDS.
constexpr int kBitmapWords = kMaxCand / 32;
static_assert(kBitmapWords == kWave, "one bitmap word per lane");
__device__ void group_union(const int* sel, unsigned* bits, int G, int per,
                            bool masks, int* uni, int* ucnt) {
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
    // this lane's word of every head's map, read once (the per-bit head
    // masks below then need no LDS reads)
    uint32_t wv[kMaxG];
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) wv[g] = g < nmaps ? bits[g * kBitmapWords + tid] : 0u;
    uint32_t word = 0u;
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) word |= wv[g];
    const int pc = __popc(word);
    // exclusive prefix sum of the popcounts over the 64 lanes
    int incl = pc;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int o = __shfl_up(incl, d);
      if (tid >= d) incl += o;
    }
    int pos = incl - pc;
    while (word) {
      const int bit = __ffs(word) - 1;
      unsigned m = kAllHeads;
      if (masks) {
        m = 0u;
#pragma unroll
        for (int g = 0; g < kMaxG; ++g) m |= ((wv[g] >> bit) & 1u) << g;
      }
      uni[pos++] = (tid * 32 + bit) | (int)(m << kUniIdBits);
      word &= word - 1u;
    }
    if (tid == kWave - 1) *ucnt = incl;
  }
}

// ---------------------------------------------------------------------------
// k_score: a[h][s] = phi(q_h) . summ[s], Eq. 6
// ---------------------------------------------------------------------------
// Workgroup = 1, 2 or 4 waves x (16 * RB) summary rows of one (b, kv head)
// (fewer waves per workgroup when that spreads a small call over more CUs;
// the waves are independent). Lane l holds FPL = n / 64 features of phi(q)
// for the G heads of the group, in chunks of at most 8 (n = 1024 and 2048
// take 2 and 4 chunks, so the rows of a batch fit in registers); each chunk
// of a row is one contiguous wave load, and all of a batch's rows are loaded
// before any is reduced. A 16-row batch is transpose-reduced inside each
// 16-lane row with DPP, then summed over the four rows.
template <int N, int G>
__global__ __launch_bounds__(256) void k_score(const float* __restrict__ phiq,
                                               const float* __restrict__ summ,
                                               float* __restrict__ scores,
                                               int Hq, int Hkv, SeqArgs sa,
                                               int64_t s_cap, int nc_cap) {
  constexpr int FPL = N / 64;
  // features per lane per chunk: all of them up to n = 512; above, 8 (4
  // for G >= 4, whose accumulators take more registers)
  constexpr int FC = FPL <= 8 ? FPL : (G >= 4 ? 4 : 8);
  constexpr int NCH = FPL / FC;            // chunks (1 for n <= 512)
  constexpr int RB = N <= 256 ? 2 : 1;     // 16-row batches per wave
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int n_cand = seq_span(sa, b).n_cand;
  const int wrow0 = (blockIdx.x * (blockDim.x >> 6) + wave) * (16 * RB);
  if (wrow0 >= n_cand) return;             // wave-uniform; no barriers below

  // chunk ch holds features ch * 64 * FC + lane * FC + e (e < FC) of lane
  // `lane`, so each chunk of a row is one contiguous 64 * FC * 4-byte wave
  // load; with one chunk (n <= 512) lane l holds features l * FPL .. + FPL
  const float* base = summ + (bh * s_cap) * N + lane * FC;
  // per row and head a running dot product over the chunks
  float part[RB][G][16];
#pragma unroll
  for (int bt = 0; bt < RB; ++bt)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) part[bt][g][r] = 0.f;
#pragma unroll 1
  for (int ch = 0; ch < NCH; ++ch) {     // one chunk's rows live at a time
    float pq[G][FC];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* src = phiq + ((b * Hq + hk * G + g) * N) + ch * 64 * FC + lane * FC;
#pragma unroll
      for (int e = 0; e < FC; ++e) pq[g][e] = src[e];
    }
    float x[RB][16][FC];
#pragma unroll
    for (int bt = 0; bt < RB; ++bt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = min(wrow0 + bt * 16 + r, n_cand - 1);
        const float* src = base + (int64_t)row * N + ch * 64 * FC;
        if constexpr (FC % 4 == 0) {
#pragma unroll
          for (int e = 0; e < FC; e += 4) {
            const float4 v = ld_stream_f4(src + e);
            x[bt][r][e] = v.x; x[bt][r][e + 1] = v.y;
            x[bt][r][e + 2] = v.z; x[bt][r][e + 3] = v.w;
          }
        } else if constexpr (FC == 2) {
          const float2 v = *reinterpret_cast<const float2*>(src);
          x[bt][r][0] = v.x; x[bt][r][1] = v.y;
        } else {
          x[bt][r][0] = src[0];
        }
      }
    // with several chunks the compiler would sink each load to its first
    // use and wait on one load at a time; keep the chunk's loads together
    if constexpr (NCH > 1) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int bt = 0; bt < RB; ++bt)
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float a = part[bt][g][r];
#pragma unroll
          for (int e = 0; e < FC; ++e) a = fmaf(x[bt][r][e], pq[g][e], a);
          part[bt][g][r] = a;
        }
  }
#pragma unroll
  for (int bt = 0; bt < RB; ++bt) {
    const int row = wrow0 + bt * 16 + (lane & 15);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      transpose_reduce<16>(part[bt][g], lane);
      float v = part[bt][g][0];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16 && row < n_cand)
        scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + row] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// k_topk_union: top-k of every query head, union per kv head
// ---------------------------------------------------------------------------
// One workgroup per (b, kv head); wave w takes heads w, w + 4, ... of the
// group. The heads' sorted selections go to LDS and the union of the group
// (ascending ids) to the workspace for the attention stage.
__global__ __launch_bounds__(256) void k_topk_union(
    const float* __restrict__ scores, int Hq, int Hkv, int G, SeqArgs sa,
    int nc_cap, int per_head, int* __restrict__ uni, int* __restrict__ ucnt,
    int umax, int32_t* __restrict__ selected, float* __restrict__ sel_scores,
    AppendArgs ap, int64_t cap) {
  __shared__ int sel_lds[kMaxG * kMaxK];
  __shared__ unsigned bits_lds[kMaxG * kBitmapWords];
  __shared__ unsigned hist_lds[4][256];
  __shared__ u64 list_lds[4][kMaxK];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.x;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  // the append of radar_append_decode (the attention kernel that reads the
  // row runs after this one)
  if (ap.K && wave == 3) append_row(ap, cap, bh, Hkv, lane);
  const Span sp = seq_span(sa, b);
  const int n_cand = sp.n_cand, k_eff = sp.k_eff, k = sa.k;
  const int npl = (n_cand + 63) / 64;
  unsigned* hist = hist_lds[wave];
  u64* list = list_lds[wave];
  for (int hl = wave; hl < G; hl += 4) {
    const int64_t hq = hk * G + hl;
    const float* src = scores + (b * Hq + hq) * (int64_t)nc_cap;
    int32_t* so = selected ? selected + (b * Hq + hq) * (int64_t)k : nullptr;
    float* sco = sel_scores ? sel_scores + (b * Hq + hq) * (int64_t)k : nullptr;
    int* row = sel_lds + hl * k_eff;
    if (npl <= 1) head_topk<1>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 2) head_topk<2>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 4) head_topk<4>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 8) head_topk<8>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 16) head_topk<16>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else head_topk<32>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
  }
  __syncthreads();
  group_union(sel_lds, bits_lds, G, k_eff, per_head != 0, uni + bh * umax,
              ucnt + bh);
}

// ---------------------------------------------------------------------------
// k_segment_mass: exact segment attention mass, ln(beta_s) per query head
// ---------------------------------------------------------------------------
// beta_s = sum over the keys of segment s of exp(q . k / sqrt(d)) (the
// segment's unnormalised attention weight; selecting its top-k is the exact
// segment search). One wave per candidate segment: the logits of each
// <= 64-token tile come from the same row-contiguous loads and
// transpose-reduce as the attention tiles, and an online log-sum-exp in
// base 2 carries across the segment's tiles. Writes ln(beta_s) to
// scores[b][h][s].
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void k_segment_mass(
    const T* __restrict__ q, const T* __restrict__ K, float* __restrict__ scores,
    int Hq, int Hkv, int64_t cap, SeqArgs sa, int nc_cap, float qscale) {
  constexpr int EPL = Elem<T>::kPer16;
  constexpr int LPR = D / EPL;
  constexpr int RPI = kWave / LPR;
  constexpr int ITER = kTile / RPI;
  constexpr float kLn2 = 0.69314718055994530942f;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int c = sa.c;
  const int s = blockIdx.x * 4 + wave;
  if (s >= seq_span(sa, b).n_cand) return; // wave-uniform; no barriers below
  const int r = lane / LPR, jj = lane % LPR;

  float qf[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 u = *reinterpret_cast<const uint4*>(
        q + ((b * Hq + hk * G + g) * D + jj * EPL));
    unpack16<T>(u, qf[g]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[g][e] *= qscale;
  }
  float m[G], l[G];
#pragma unroll
  for (int g = 0; g < G; ++g) { m[g] = -INFINITY; l[g] = 0.f; }

  for (int off = 0; off < c; off += kTile) {
    const int len = min(kTile, c - off);
    const T* kbase = K + (bh * cap + (int64_t)s * c + off) * D + jj * EPL;
    uint4 kr[ITER];
#pragma unroll
    for (int i = 0; i < ITER; ++i)
      kr[i] = ld_stream(kbase + (int64_t)min(i * RPI + r, len - 1) * D);
    float pl[G][ITER];
#pragma unroll
    for (int i = 0; i < ITER; ++i) {
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
    const bool mine_ok = (jj * RPI + r) < len;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      transpose_reduce<LPR>(pl[g], lane);
      const float lg = pl[g][0];
      const float mt = wave_max(mine_ok ? lg : -INFINITY);
      const float mn = fmaxf(m[g], mt);
      const float p = mine_ok ? fast_exp2(lg - mn) : 0.f;
      l[g] = fmaf(l[g], fast_exp2(m[g] - mn), wave_sum(p));
      m[g] = mn;
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
      scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + s] = (m[g] + __log2f(l[g])) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// k_union_given: union of caller-given selections (attention on a supplied
// selection, the last step of Algorithm 1 alone)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_union_given(
    const int32_t* __restrict__ given, int given_k, int Hq, int Hkv, int G,
    SeqArgs sa, int per_head, int* __restrict__ uni, int* __restrict__ ucnt,
    int umax) {
  __shared__ int sel_lds[kMaxG * kMaxK];
  __shared__ unsigned bits_lds[kMaxG * kBitmapWords];
  const int64_t bh = blockIdx.x;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int n_cand = seq_span(sa, b).n_cand;
  const int M = G * given_k;
  for (int i = threadIdx.x; i < M; i += 256) {
    const int hl = i / given_k, r = i % given_k;
    const int id = given[(b * Hq + hk * G + hl) * (int64_t)given_k + r];
    sel_lds[i] = (id >= 0 && id < n_cand) ? id : -1;
  }
  __syncthreads();
  group_union(sel_lds, bits_lds, G, given_k, per_head != 0, uni + bh * umax,
              ucnt + bh);
}

// ---------------------------------------------------------------------------
// exact attention over <= 64-token tiles (shared by k_attend and k_decode_fused)
// ---------------------------------------------------------------------------
// The attended tokens of a (b, kv head) are cut into tiles of <= 64 tokens
// that never cross a segment or the window boundary. A wave processes one
// tile at a time: lane (r, jj) (r = lane / LPR) reads the 16-byte chunk jj of
// rows r, r + RPI, ... so every load instruction covers RPI whole rows
// contiguously (rows past the tile end re-read its last row and are masked).
// q.k partials are transpose-reduced so that each lane ends with one token's
// logit, softmax runs across the wave, and p is broadcast back (DPP row
// broadcast) to the lanes that hold the matching V chunks. The state carries
// across tiles as an online softmax: running max m and sum l (log2 units,
// wave-uniform) and unreduced per-lane accumulators.
template <typename T, int D, int G>
struct TileAttn {
  static constexpr int EPL = Elem<T>::kPer16;   // elements per 16-byte chunk
  static constexpr int LPR = D / EPL;           // lanes per row
  static constexpr int RPI = kWave / LPR;       // rows per load instruction
  static constexpr int ITER = kTile / RPI;      // load instructions per tile
  static_assert(ITER == LPR, "tile shape");

  float qf[G][EPL];
  float m[G], l[G], acc[G][EPL];

  // q0: the group's first query head; qscale folds log2(e) / sqrt(d)
  __device__ __forceinline__ void init(const T* __restrict__ q0, float qscale,
                                       int lane) {
    const int jj = lane % LPR;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint4 u = *reinterpret_cast<const uint4*>(q0 + g * D + jj * EPL);
      unpack16<T>(u, qf[g]);
#pragma unroll
      for (int e = 0; e < EPL; ++e) qf[g][e] *= qscale;
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
    const T* kbase = K + row0 * D + jj * EPL;
    const T* vbase = V + row0 * D + jj * EPL;
    uint4 kr[ITER], vr[ITER];
#pragma unroll
    for (int i = 0; i < ITER; ++i)
      kr[i] = ld_stream(kbase + (int64_t)min(i * RPI + r, len - 1) * D);
#pragma unroll
    for (int i = 0; i < ITER; ++i)
      vr[i] = ld_stream(vbase + (int64_t)min(i * RPI + r, len - 1) * D);

    // logits: lane (r, jj) ends with the logit of tile row jj * RPI + r
    float lg[G];
    {
      float pl[G][ITER];
#pragma unroll
      for (int i = 0; i < ITER; ++i) {
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
#pragma unroll
      for (int g = 0; g < G; ++g) {
        transpose_reduce<LPR>(pl[g], lane);
        lg[g] = pl[g][0];
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
#pragma unroll
    for (int msk = LPR; msk < kWave; msk <<= 1)
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] += __shfl_xor(acc[g][e], msk);
  }
};

// ---------------------------------------------------------------------------
// k_attend: split attention, one partial (max, sum, acc[d]) per workgroup
// ---------------------------------------------------------------------------
// Tiles of a (b, kv head): tiles_per_seg per union segment, then ceil(|W| /
// 64) window tiles, then ceil(sinks / 64) sink tiles. Workgroup j takes
// tiles [4 tpw j, 4 tpw (j + 1)); wave w takes every fourth of them from
// 4 tpw j + w, with an online softmax across its tiles, and the workgroup
// merges its four waves in LDS. With per_head set, a segment tile counts
// only for the heads that selected the segment.
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void k_attend(
    const T* __restrict__ q, const T* __restrict__ K, const T* __restrict__ V,
    const int* __restrict__ uni, const int* __restrict__ ucnt,
    float* __restrict__ part, int Hq, int Hkv, int64_t cap,
    int tiles_per_seg, SeqArgs sa, int per_head, int umax, int maxwg, int tpw,
    float qscale) {
  using TA = TileAttn<T, D, G>;
  constexpr int EPL = TA::EPL, LPR = TA::LPR;
  constexpr int PSTRIDE = D + 4;

  __shared__ float wm[4][G], wl[4][G];
  __shared__ __attribute__((aligned(16))) float wacc[4][G][D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int j = blockIdx.x;
  const Span sp = seq_span(sa, b);
  const int c = sa.c;

  const int U = ucnt[bh];
  const int seg_tiles = U * tiles_per_seg;
  const int win_tiles = (int)(((int64_t)sp.t - sp.ws + kTile - 1) / kTile);
  const int total = seg_tiles + win_tiles + (sp.sink + kTile - 1) / kTile;
  const int nwg = (total + 4 * tpw - 1) / (4 * tpw);
  if (j >= nwg) return;

  TA ta;
  ta.init(q + (b * Hq + hk * G) * D, qscale, lane);
  const int t_end = min(total, (j + 1) * 4 * tpw);
  for (int ti = j * 4 * tpw + wave; ti < t_end; ti += 4) {   // wave-uniform
    int64_t start;
    int len;
    unsigned hm = kAllHeads;
    if (ti < seg_tiles) {
      const int e = uni[bh * umax + ti / tiles_per_seg];
      const int s = e & ((1 << kUniIdBits) - 1);
      if (per_head) hm = (unsigned)e >> kUniIdBits;
      const int off = (ti % tiles_per_seg) * kTile;
      start = (int64_t)s * c + off;
      len = min(kTile, c - off);
    } else if (ti < seg_tiles + win_tiles) {
      start = sp.ws + (int64_t)(ti - seg_tiles) * kTile;
      len = (int)min((int64_t)kTile, sp.t - start);
    } else {
      const int off = (ti - seg_tiles - win_tiles) * kTile;
      start = (int64_t)off - sa.n_sink;
      len = min(kTile, sp.sink - off);
    }
    ta.tile(K, V, bh * cap + start, len, lane, hm);
  }
  ta.reduce_rows();

  const int jj = lane % LPR;
  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) wacc[wave][g][jj * EPL + e] = ta.acc[g][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = ta.m[g]; wl[wave][g] = ta.l[g]; }
  }
  __syncthreads();

  float* pj = part + ((bh * maxwg + j) * G) * (int64_t)PSTRIDE;
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    float M = wm[0][g];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, wm[w][g]);
    float a = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = wm[w][g] == -INFINITY ? 0.f : fast_exp2(wm[w][g] - M);
      a = fmaf(wacc[w][g][e], f, a);
      L = fmaf(wl[w][g], f, L);
    }
    pj[g * PSTRIDE + 4 + e] = a;
    if (e == 0) { pj[g * PSTRIDE] = M; pj[g * PSTRIDE + 1] = L; }
  }
}

// ---------------------------------------------------------------------------
// k_decode_fused: the whole decode step of one (b, kv head) in R workgroups
// ---------------------------------------------------------------------------
// Every workgroup of a pair runs the whole selection itself (phases 1-4 give
// the same result in each: the same inputs, the same order of operations),
// so no stage hands data to another workgroup (the per-XCD L2s are not
// coherent, so a cross-workgroup hand-off would need a kernel boundary or a
// cache flush). With R = 1 (at least as many pairs as compute units) one
// 512-thread workgroup per pair keeps every CU streaming and writes the
// output; with fewer pairs R workgroups share a pair's attention tiles and
// each writes a partial that k_combine merges (the repeated summary reads
// mostly hit the caches). Phases:
//   1. phi(q) of the group's G heads into LDS (16 lanes per Omega row;
//      Omega in fp32 or bf16, obf), with each wave's first summary rows
//      already in flight (waves whose first row is past the candidates
//      load none);
//   2. Eq. 6 scores of all candidates into LDS (16 or 32 summary rows per
//      wave per pass, streaming loads; above n = 512 each 16-row batch in
//      feature chunks, and phase 1 writes phi(q) to LDS chunk by chunk);
//   3. waves < G take the top-k of one head each, while the other waves
//      already attend the window tiles (the window never depends on the
//      selection);
//   4. the group's union in LDS;
//   5. every wave attends segment tiles (tile i to workgroup i mod R, and
//      in it to wave (i / R) mod 8);
//   6. the waves' online-softmax states merge in LDS into the output (or
//      the workgroup's partial).
// With SEL set the kernel stops after phase 4 and writes the union to
// uni_out / ucnt_out for the split path's attention (the select path: one
// workgroup per pair replaces the phi(q), score and top-k kernels).
constexpr int kFusedWaves = 8;
constexpr int kFusedMaxG = 4;
constexpr int kFusedMaxCand = 1024;

template <typename T, int D, int G, int N, bool SEL>
__global__ __launch_bounds__(512) void k_decode_fused(
    const T* __restrict__ q, const T* __restrict__ K, const T* __restrict__ V,
    const void* __restrict__ omega, bool obf, const float* __restrict__ summ,
    T* __restrict__ out, int32_t* __restrict__ selected,
    float* __restrict__ sel_scores, int Hq, int Hkv, int64_t cap,
    int64_t s_cap, int tiles_per_seg, SeqArgs sa, int per_head, float s1,
    float s2, float inv_sqrt_n, float qscale, int* __restrict__ uni_out,
    int* __restrict__ ucnt_out, int umax, AppendArgs ap, int R, int n_pairs,
    float* __restrict__ part, int maxwg) {
  constexpr int NW = kFusedWaves;
  constexpr int QPL = D / 16;              // q elements per lane (phase 1)
  constexpr int FPL = N / 64;              // features per lane (phase 2)
  using TA = TileAttn<T, D, G>;
  constexpr int EPL = TA::EPL, LPR = TA::LPR;
  constexpr int SEL_FLOATS = G * N + G * kFusedMaxCand;
  constexpr int MRG_FLOATS = NW * G * D;
  constexpr int AREA = SEL_FLOATS > MRG_FLOATS ? SEL_FLOATS : MRG_FLOATS;
  static_assert(G <= kFusedMaxG, "group");
  static_assert(N % (4 * NW) == 0, "features");

  // phi(q) and the scores live only until the top-k; the merge reuses them
  __shared__ __attribute__((aligned(16))) float area[AREA];
  __shared__ int sel_lds[G * kMaxK];
  __shared__ unsigned bits_lds[G * kBitmapWords];
  __shared__ int uni_lds[G * kMaxK];
  __shared__ unsigned hist_lds[G][256];
  __shared__ u64 list_lds[G][kMaxK];
  __shared__ float wm[NW][G], wl[NW][G];
  __shared__ int ucnt_lds;
  float* phq = area;                       // [G][N]
  float* sc = area + G * N;                // [G][kFusedMaxCand]
  float* wacc = area;                      // [NW][G][D]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // workgroup rj < R of pair bh: the workgroups of a pair differ by a
  // multiple of n_pairs, so they share an XCD (and its L2) when n_pairs is a
  // multiple of 8
  const int64_t bh = blockIdx.x % n_pairs;
  const int rj = (int)(blockIdx.x / n_pairs);
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const T* q0 = q + (b * Hq + hk * G) * D;
  const Span sp = seq_span(sa, b);
  const int c = sa.c, k = sa.k, n_cand = sp.n_cand, k_eff = sp.k_eff;
  const int64_t ws = sp.ws, t = sp.t;

  // The append of radar_append_decode: the last wave writes the pair's new
  // row before anything reads it. The row belongs to the window (never to a
  // candidate segment), read from phase 3 on, after a barrier: those of
  // phases 1 and 2, or this one when there are no candidates.
  if (ap.K) {                              // uniform
    if (wave == NW - 1) append_row(ap, cap, bh, Hkv, lane);
    if (n_cand == 0) __syncthreads();
  }

  if (n_cand > 0) {                        // uniform
    // Each wave's first batch of summary rows goes in flight before phi(q)
    // is computed (the rows do not depend on it), so the projection's
    // latency overlaps the stream of the scores.
    constexpr int RB = FPL <= 4 ? 2 : 1;   // 16-row batches per pass
    const float* base = summ + (bh * s_cap) * N + lane * FPL;
    float x[RB][16][FPL];
    auto load_rows = [&](int rb) {
#pragma unroll
      for (int bt = 0; bt < RB; ++bt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int row = min(rb + bt * 16 + i, n_cand - 1);
          const float* src = base + (int64_t)row * N;
          if constexpr (FPL % 4 == 0) {
#pragma unroll
            for (int e = 0; e < FPL; e += 4) {
              const float4 v = ld_stream_f4(src + e);
              x[bt][i][e] = v.x; x[bt][i][e + 1] = v.y;
              x[bt][i][e + 2] = v.z; x[bt][i][e + 3] = v.w;
            }
          } else if constexpr (FPL == 2) {
            const float2 v = *reinterpret_cast<const float2*>(src);
            x[bt][i][0] = v.x; x[bt][i][1] = v.y;
          } else {
            x[bt][i][0] = src[0];
          }
        }
    };

    // ---- 1. phi(q) -----------------------------------------------------
    // 16 lanes per Omega row, 4 rows per wave and pass, NP passes. All of a
    // chunk's Omega loads are issued before any is used, then the summary
    // rows (when they fit in registers next to them), then the dots. The
    // phase is compiled once per Omega storage type (BF: bf16) and one copy
    // runs, so both kinds of load stay in flight together.
    const int rb0 = wave * 16 * RB;
    auto phase1 = [&](auto bf_tag) {
      constexpr bool BF = decltype(bf_tag)::value;
      constexpr int NP = N / (4 * NW);       // passes
      constexpr int PC = NP < 8 ? NP : 8;    // passes per load chunk
      constexpr bool kPrefetch = NP <= 8;
      const int r = lane >> 4, jj = lane & 15;
      float qv[G][QPL], nrm[G];
      // above n = 512 each chunk's features go to LDS at once (all NP
      // passes would not fit in registers)
      constexpr bool kChunkOut = N > 512;
      float ph[kChunkOut ? PC : NP][G];
#pragma unroll
      for (int c0 = 0; c0 < NP; c0 += PC) {
        // the Omega loads come first in each copy of the phase, so the
        // compiler cannot hoist the q loads and their conversion (code the
        // two copies share) above the choice of copy, where they would
        // have to be waited for
        uint4 om[PC][QPL / 4];
        load_omega_rows<BF, PC, QPL>(om, omega, [&](int p) {
          return (int64_t)((c0 + p) * 4 * NW + wave * 4 + r) * D + jj * QPL;
        });
        if (c0 == 0) {
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < QPL; ++e) qv[g][e] = to_f32<T>(q0[g * D + jj * QPL + e]);
        }
        // rows clamp to the last candidate; a wave whose first row is past
        // it has no rows (the candidate count is uniform)
        if (kPrefetch && c0 == 0 && rb0 < n_cand) load_rows(rb0);
        if (c0 == 0) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float sq = 0.f;
#pragma unroll
            for (int e = 0; e < QPL; ++e) sq = fmaf(qv[g][e], qv[g][e], sq);
            nrm[g] = row_sum(sq);
          }
        }
#pragma unroll
        for (int p = 0; p < PC; ++p) {
          float a[G];
#pragma unroll
          for (int g = 0; g < G; ++g) a[g] = 0.f;
#pragma unroll
          for (int e4 = 0; e4 < QPL / 4; ++e4) {
            float4 o = omega_f4<BF>(om[p][e4]);
            if constexpr (sizeof(T) == 2 && !BF) {
              o.x = round_bf16(o.x); o.y = round_bf16(o.y);
              o.z = round_bf16(o.z); o.w = round_bf16(o.w);
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
              a[g] = fmaf(o.x, qv[g][4 * e4], a[g]);
              a[g] = fmaf(o.y, qv[g][4 * e4 + 1], a[g]);
              a[g] = fmaf(o.z, qv[g][4 * e4 + 2], a[g]);
              a[g] = fmaf(o.w, qv[g][4 * e4 + 3], a[g]);
            }
          }
#pragma unroll
          for (int g = 0; g < G; ++g)
            ph[kChunkOut ? p : c0 + p][g] =
                fast_exp2(fmaf(row_sum(a[g]), s1, -nrm[g] * s2)) * inv_sqrt_n;
        }
        if constexpr (kChunkOut) {
          if (jj == 0) {
#pragma unroll
            for (int p = 0; p < PC; ++p)
#pragma unroll
              for (int g = 0; g < G; ++g)
                phq[g * N + (c0 + p) * 4 * NW + wave * 4 + r] = ph[p][g];
          }
        }
      }
      if constexpr (!kChunkOut) {
        if (!kPrefetch && rb0 < n_cand) load_rows(rb0);
        if (jj == 0) {
#pragma unroll
          for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int g = 0; g < G; ++g) phq[g * N + p * 4 * NW + wave * 4 + r] = ph[p][g];
        }
      }
    };
    if constexpr (sizeof(T) == 2) {
      if (obf) phase1(std::true_type{});
      else phase1(std::false_type{});
    } else {
      phase1(std::false_type{});
    }
    __syncthreads();

    // ---- 2. scores ------------------------------------------------------
    if constexpr (N > 512) {
      // each 16-row batch in chunks of FC features per lane (chunk ch of
      // lane l: features ch * 64 * FC + l * FC + e), the layout and order
      // of the split path's score kernel, so a lane holds one chunk of the
      // batch's rows at a time
      constexpr int FC = G >= 4 ? 4 : 8;
      constexpr int NCH = FPL / FC;
      const float* rbase = summ + (bh * s_cap) * N + lane * FC;
      for (int rb = wave * 16; rb < n_cand; rb += NW * 16) {
        float part[G][16];
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int i = 0; i < 16; ++i) part[g][i] = 0.f;
#pragma unroll 1
        for (int ch = 0; ch < NCH; ++ch) {
          float xx[16][FC];
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int row = min(rb + i, n_cand - 1);
            const float* src = rbase + (int64_t)row * N + ch * 64 * FC;
#pragma unroll
            for (int e = 0; e < FC; e += 4) {
              const float4 v = ld_stream_f4(src + e);
              xx[i][e] = v.x; xx[i][e + 1] = v.y; xx[i][e + 2] = v.z; xx[i][e + 3] = v.w;
            }
          }
          float pq[G][FC];
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < FC; ++e) pq[g][e] = phq[g * N + ch * 64 * FC + lane * FC + e];
          // keep the chunk's loads together (the compiler would otherwise
          // sink each to its first use and wait on one at a time)
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              float a = part[g][i];
#pragma unroll
              for (int e = 0; e < FC; ++e) a = fmaf(xx[i][e], pq[g][e], a);
              part[g][i] = a;
            }
        }
        const int row = rb + (lane & 15);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          transpose_reduce<16>(part[g], lane);
          float v = part[g][0];
          v += __shfl_xor(v, 16);
          v += __shfl_xor(v, 32);
          if (lane < 16 && row < n_cand) sc[g * kFusedMaxCand + row] = v;
        }
      }
    } else {
      float pq[G][FPL];
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < FPL; ++e) pq[g][e] = phq[g * N + lane * FPL + e];
      for (int rb = rb0; rb < n_cand; rb += NW * 16 * RB) {
        if (rb != rb0) load_rows(rb);
#pragma unroll
        for (int bt = 0; bt < RB; ++bt) {
          const int row = rb + bt * 16 + (lane & 15);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float part[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              float a = 0.f;
#pragma unroll
              for (int e = 0; e < FPL; ++e) a = fmaf(x[bt][i][e], pq[g][e], a);
              part[i] = a;
            }
            transpose_reduce<16>(part, lane);
            float v = part[0];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            if (lane < 16 && row < n_cand) sc[g * kFusedMaxCand + row] = v;
          }
        }
      }
    }
    __syncthreads();
  }

  // ---- 3. top-k (waves < G) | window and sink tiles (the other waves) ----
  TA ta;
  if constexpr (!SEL) ta.init(q0, qscale, lane);
  const int win_tiles = (int)((t - ws + kTile - 1) / kTile);
  const int extra_tiles = win_tiles + (sp.sink + kTile - 1) / kTile;
  if (wave < G) {
    const int64_t hq = hk * G + wave;
    // every workgroup of the pair selects the same segments; the first
    // one reports them
    int32_t* so = selected && rj == 0 ? selected + (b * Hq + hq) * (int64_t)k : nullptr;
    float* sco = sel_scores && rj == 0 ? sel_scores + (b * Hq + hq) * (int64_t)k : nullptr;
    const float* src = sc + wave * kFusedMaxCand;
    int* row = sel_lds + wave * k_eff;
    unsigned* hist = hist_lds[wave];
    u64* list = list_lds[wave];
    const int npl = (n_cand + 63) / 64;
    if (npl <= 1) head_topk<1>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 2) head_topk<2>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 4) head_topk<4>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else if (npl <= 8) head_topk<8>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
    else head_topk<16>(src, n_cand, k, k_eff, row, so, sco, lane, hist, list);
  } else if constexpr (!SEL) {
    for (int i = rj + (wave - G) * R; i < extra_tiles; i += (NW - G) * R) {
      int64_t start;
      int len;
      if (i < win_tiles) {
        start = ws + (int64_t)i * kTile;
        len = (int)min((int64_t)kTile, t - start);
      } else {
        const int off = (i - win_tiles) * kTile;
        start = (int64_t)off - sa.n_sink;
        len = min(kTile, sp.sink - off);
      }
      ta.tile(K, V, bh * cap + start, len, lane, kAllHeads);
    }
  }
  __syncthreads();

  // ---- 4. union -----------------------------------------------------------
  // With one query head per group its selection is the set to attend (in
  // score order; the online softmax does not depend on the order), so the
  // bitmap union is skipped.
  const int* segs = sel_lds;
  int n_segs = k_eff;
  if constexpr (G > 1 || SEL) {
    group_union(sel_lds, bits_lds, G, k_eff, per_head != 0, uni_lds, &ucnt_lds);
    __syncthreads();
    segs = uni_lds;
    n_segs = ucnt_lds;
  }
  if constexpr (SEL) {                     // hand the union to the split path
    for (int i = tid; i < n_segs; i += NW * 64) uni_out[bh * umax + i] = segs[i];
    if (tid == 0) ucnt_out[bh] = n_segs;
    return;
  }
  const int seg_tiles = n_segs * tiles_per_seg;

  // ---- 5. segment tiles ---------------------------------------------------
  for (int i = rj + wave * R; i < seg_tiles; i += NW * R) {
    const int e = segs[i / tiles_per_seg];
    const int s = e & ((1 << kUniIdBits) - 1);
    // (the plain selection of a one-head group carries no head mask)
    const unsigned hm = (G > 1 && per_head) ? (unsigned)e >> kUniIdBits : kAllHeads;
    const int off = (i % tiles_per_seg) * kTile;
    ta.tile(K, V, bh * cap + (int64_t)s * c + off, min(kTile, c - off), lane, hm);
  }

  // ---- 6. merge -----------------------------------------------------------
  ta.reduce_rows();
  __syncthreads();                         // phq / sc are dead from here on
  const int jj = lane % LPR;
  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e)
        wacc[(wave * G + g) * D + jj * EPL + e] = ta.acc[g][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = ta.m[g]; wl[wave][g] = ta.l[g]; }
  }
  __syncthreads();
  for (int x = tid; x < G * D; x += NW * 64) {
    const int g = x / D, e = x % D;
    float M = wm[0][g];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w][g]);
    float a = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = wm[w][g] == -INFINITY ? 0.f : fast_exp2(wm[w][g] - M);
      a = fmaf(wacc[(w * G + g) * D + e], f, a);
      L = fmaf(wl[w][g], f, L);
    }
    if (R == 1) {
      const float o = !sp.ok ? __uint_as_float(0x7fc00000u) : (L > 0.f ? a / L : 0.f);
      out[(b * Hq + hk * G + g) * D + e] = from_f32<T>(o);
    } else {                               // partial of this workgroup's tiles
      float* pj = part + ((bh * maxwg + rj) * G + g) * (int64_t)(D + 4);
      pj[4 + e] = a;
      if (e == 0) { pj[0] = M; pj[1] = L; }
    }
  }
}

// ---------------------------------------------------------------------------
// k_combine: log-sum-exp merge of the partials of each (b, q head)
// ---------------------------------------------------------------------------
// Grid (B * Hq, D / DS), NT threads: each workgroup produces DS output dims
// of one query head from at most MAXP partials. Every workgroup takes the
// maximum and the scaled sum over all the head's partials (a (max, sum)
// pair each, kept in registers between the passes); then the NT / DS groups
// of threads sum disjoint subsets of the partials' accumulators over its
// dims, and LDS adds the groups.
// With many partials per head (DS = 32, MAXP = kMaxWg) a head's partials are
// read by several CUs at once, and each thread issues its first PF
// accumulator loads before the first reduction, so most of the merge waits
// on memory once. With few (DS = D, PF = 0) one workgroup per head saves the
// launches, and the accumulators are read after the reductions.
template <typename T, int D, int NT, int DS, int MAXP, int PF>
__global__ __launch_bounds__(NT) void k_combine(
    const float* __restrict__ part, const int* __restrict__ ucnt,
    T* __restrict__ out, int Hq, int Hkv, int G, int tiles_per_seg,
    SeqArgs sa, int maxwg, int tpw, int fixed_nwg) {
  constexpr int PSTRIDE = D + 4;
  constexpr int NWAVE = NT / kWave;
  constexpr int NGRP = NT / DS;            // thread groups over the partials
  constexpr int PPT = (MAXP + NT - 1) / NT;  // (max, sum) pairs per thread
  static_assert(D % DS == 0 && MAXP <= kMaxWg && PF * NGRP <= MAXP, "shape");
  __shared__ float f_lds[MAXP];
  __shared__ float red_lds[2 * NWAVE];
  __shared__ float acc_lds[NT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bhq = blockIdx.x;
  const int e0 = blockIdx.y * DS;
  const int64_t b = bhq / Hq, hq = bhq % Hq;
  const int64_t hk = hq / G;
  const int g = (int)(hq % G);
  const int64_t bh = b * Hkv + hk;
  const Span sp = seq_span(sa, b);
  // partials of the pair: fixed_nwg (one per workgroup of the fused
  // kernel), or one per 4 tpw tiles of the split attention; the host sizes
  // MAXP from the same bound
  int nwg = fixed_nwg;
  if (nwg == 0) {
    const int extra = (int)(((int64_t)sp.t - sp.ws + kTile - 1) / kTile) +
                      (sp.sink + kTile - 1) / kTile;
    nwg = (ucnt[bh] * tiles_per_seg + extra + 4 * tpw - 1) / (4 * tpw);
  }
  nwg = min(nwg, MAXP);
  T* o = out + bhq * D + e0;
  if (!sp.ok || nwg == 0) {                // invalid length / nothing attended
    if (tid < DS) o[tid] = from_f32<T>(sp.ok ? 0.f : __uint_as_float(0x7fc00000u));
    return;
  }
  const float* pb = part + ((bh * maxwg) * G + g) * (int64_t)PSTRIDE;
  const int64_t wstride = (int64_t)G * PSTRIDE;

  float mw[PPT], lw[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int w = tid + i * NT;
    mw[i] = w < nwg ? pb[w * wstride] : -INFINITY;
    lw[i] = w < nwg ? pb[w * wstride + 1] : 0.f;
  }
  const int e = tid % DS, grp = tid / DS;
  const float* pe = pb + 4 + e0 + e;
  float av[PF > 0 ? PF : 1];
#pragma unroll
  for (int j = 0; j < PF; ++j) {
    const int w = grp + j * NGRP;
    av[j] = w < nwg ? pe[w * wstride] : 0.f;
  }

  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < PPT; ++i) mx = fmaxf(mx, mw[i]);
  mx = wave_max(mx);
  if (lane == 0) red_lds[wave] = mx;
  __syncthreads();
  float M = red_lds[0];
#pragma unroll
  for (int i = 1; i < NWAVE; ++i) M = fmaxf(M, red_lds[i]);
  if (M == -INFINITY) {                    // this head attended nothing
    if (tid < DS) o[tid] = from_f32<T>(0.f);
    return;
  }
  float ls = 0.f;
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int w = tid + i * NT;
    if (w < nwg) {
      const float f = fast_exp2(mw[i] - M);
      f_lds[w] = f;
      ls = fmaf(lw[i], f, ls);
    }
  }
  ls = wave_sum(ls);
  if (lane == 0) red_lds[NWAVE + wave] = ls;
  __syncthreads();
  float L = 0.f;
#pragma unroll
  for (int i = 0; i < NWAVE; ++i) L += red_lds[NWAVE + i];
  float a = 0.f;
#pragma unroll
  for (int j = 0; j < PF; ++j) {
    const int w = grp + j * NGRP;
    if (w < nwg) a = fmaf(av[j], f_lds[w], a);
  }
#pragma unroll 8
  for (int w = grp + PF * NGRP; w < nwg; w += NGRP) a = fmaf(pe[w * wstride], f_lds[w], a);
  acc_lds[tid] = a;
  __syncthreads();
  if (tid < DS) {
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < NGRP; ++i) sum += acc_lds[i * DS + tid];
    o[tid] = from_f32<T>(sum / L);
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
thread_local char g_last_error[256] = "";


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
thread_local Profiler g_prof;

template <typename F, typename... Args>
void launch(int kind, F kern, dim3 grid, dim3 block, size_t shm, hipStream_t st,
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

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

radar_status check_cfg(const radar_config* cfg, Shape* s) {
  if (!cfg) return RADAR_EINVAL;
  if (cfg->batch < 1 || cfg->n_q_heads < 1 || cfg->n_kv_heads < 1 ||
      cfg->seg_len < 1 || cfg->window < 0 || cfg->capacity < 1 ||
      cfg->n_q_heads % cfg->n_kv_heads != 0)
    return RADAR_EINVAL;
  if (cfg->kv_dtype != RADAR_F32 && cfg->kv_dtype != RADAR_BF16) return RADAR_EINVAL;
  if (cfg->omega_dtype != RADAR_F32 && cfg->omega_dtype != RADAR_BF16) return RADAR_EINVAL;
  // a bf16 Omega only where the projection rounds Omega to bf16
  if (cfg->omega_dtype == RADAR_BF16 && cfg->kv_dtype != RADAR_BF16) return RADAR_EINVAL;
  if (cfg->n_sink < 0 || cfg->n_sink > cfg->capacity) return RADAR_EINVAL;
  if (cfg->gqa_mode != RADAR_GQA_UNION && cfg->gqa_mode != RADAR_GQA_PER_HEAD)
    return RADAR_EINVAL;
  const int G = cfg->n_q_heads / cfg->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return RADAR_EUNSUPPORTED;
  if (cfg->head_dim != 64 && cfg->head_dim != 128) return RADAR_EUNSUPPORTED;
  const int n = cfg->n_features;
  if (n != 64 && n != 128 && n != 256 && n != 512 && n != 1024 && n != 2048)
    return RADAR_EUNSUPPORTED;
  // row counts fit int32; (b, kv head) pairs fit a grid's y dimension
  if (cfg->capacity > INT32_MAX) return RADAR_EUNSUPPORTED;
  if ((int64_t)cfg->batch * cfg->n_kv_heads > 65535) return RADAR_EUNSUPPORTED;
  s->B = cfg->batch; s->Hq = cfg->n_q_heads; s->Hkv = cfg->n_kv_heads; s->G = G;
  s->d = cfg->head_dim; s->n = n; s->c = cfg->seg_len; s->w = cfg->window;
  s->cap = cfg->capacity; s->s_cap = cfg->capacity / cfg->seg_len;
  s->dt = cfg->kv_dtype; s->n_sink = cfg->n_sink;
  s->obf = cfg->omega_dtype == RADAR_BF16;
  s->per_head = cfg->gqa_mode == RADAR_GQA_PER_HEAD;
  return RADAR_OK;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct WsLayout {
  size_t phiq, scores, uni, ucnt, part, total;
  int umax, maxwg, tiles_per_seg;
};

WsLayout ws_layout(const Shape& s, int k) {
  WsLayout L;
  L.tiles_per_seg = (int)ceil_div(s.c, kTile);
  L.umax = (int)std::max<int64_t>(1, std::min<int64_t>((int64_t)s.G * k, s.s_cap));
  const int64_t wmax = std::min<int64_t>(s.cap, (int64_t)s.w + s.c);
  const int64_t wt = ceil_div(wmax, kTile) +
                     ceil_div(std::min<int64_t>(s.n_sink, s.cap), kTile);
  L.maxwg = (int)ceil_div((int64_t)L.umax * L.tiles_per_seg + wt, 4);
  const size_t bh = (size_t)s.B * s.Hkv;
  size_t off = 0;
  L.phiq = off;        off += align256((size_t)s.B * s.Hq * s.n * 4);
  L.scores = off;      off += align256((size_t)s.B * s.Hq * std::max<int64_t>(1, s.s_cap) * 4);
  L.uni = off;         off += align256(bh * L.umax * 4);
  L.ucnt = off;        off += align256(bh * 4);
  L.part = off;        off += align256(bh * L.maxwg * s.G * (s.d + 4) * 4);
  L.total = off;
  return L;
}

radar_status launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return RADAR_OK;
  snprintf(g_last_error, sizeof g_last_error, "%s", hipGetErrorString(e));
  return RADAR_EHIP;
}

// ---- build ---------------------------------------------------------------
int g_num_cu = 0;
int num_cu() {
  if (g_num_cu == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      g_num_cu = v;
    else
      g_num_cu = 256;
  }
  return g_num_cu;
}

template <typename T, int D, int FT>
radar_status launch_build_t(const Shape& s, const void* K, const void* omega,
                            float* summ, int seg_first, int seg_count,
                            const int64_t* pos, hipStream_t st) {
  const int slices = s.n / (64 * FT);
  const int64_t items = (int64_t)s.B * s.Hkv * seg_count;
  if (items == 0) return RADAR_OK;
  if (items >= ((int64_t)1 << 31)) return RADAR_EUNSUPPORTED;   // 32-bit item ids
  auto kern = k_build<T, D, FT>;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 256, 0) != hipSuccess || per_cu < 1)
    per_cu = 1;
  (void)hipGetLastError();
  const int64_t resident = (int64_t)per_cu * num_cu();
  const int64_t gx = std::min<int64_t>(items, std::max<int64_t>(1, resident / slices));
  const float s1 = kLog2e / std::pow((float)s.d, 0.25f);
  const float s2 = kLog2e / (2.f * std::sqrt((float)s.d));
  const float out_scale = 1.f / ((float)s.c * std::sqrt((float)s.n));
  launch(RADAR_K_BUILD, kern, dim3((unsigned)gx, (unsigned)slices), dim3(256), 0, st,
                     reinterpret_cast<const T*>(K), omega, s.obf, summ, s.n, s.c, s.cap,
                     s.s_cap, seg_first, seg_count, items, s1, s2, out_scale, s.cap,
                     pos, s.Hkv, s.n_sink);
  return launch_status();
}

template <typename T, int D>
radar_status launch_build_d(const Shape& s, const void* K, const void* omega,
                            float* summ, int seg_first, int seg_count,
                            const int64_t* pos, hipStream_t st) {
  // features per workgroup = 64 * FT; FT capped so the resident Omega slice
  // stays at 128 VGPRs or fewer
  constexpr int FTMAX = (D * sizeof(T) <= 256) ? 8 : 4;
  const int ft = std::min(s.n / 64, FTMAX);
  switch (ft) {
    case 1: return launch_build_t<T, D, 1>(s, K, omega, summ, seg_first, seg_count, pos, st);
    case 2: return launch_build_t<T, D, 2>(s, K, omega, summ, seg_first, seg_count, pos, st);
    case 4: return launch_build_t<T, D, 4>(s, K, omega, summ, seg_first, seg_count, pos, st);
    default:
      if constexpr (FTMAX >= 8)
        return launch_build_t<T, D, 8>(s, K, omega, summ, seg_first, seg_count, pos, st);
      return RADAR_EUNSUPPORTED;
  }
}

// K: the first row after the sinks (after_sinks); pos: per-sequence segment
// closes (seg_first / seg_count then 0 / 1)
radar_status launch_build(const Shape& s, const void* K, const void* omega,
                          float* summ, int seg_first, int seg_count,
                          const int64_t* pos, hipStream_t st) {
  if (s.dt == RADAR_BF16)
    return s.d == 64 ? launch_build_d<bf16_t, 64>(s, K, omega, summ, seg_first, seg_count, pos, st)
                     : launch_build_d<bf16_t, 128>(s, K, omega, summ, seg_first, seg_count, pos, st);
  return s.d == 64 ? launch_build_d<float, 64>(s, K, omega, summ, seg_first, seg_count, pos, st)
                   : launch_build_d<float, 128>(s, K, omega, summ, seg_first, seg_count, pos, st);
}

// K / V rows after the n_sink sink rows of the first (b, kv head): the
// kernels address segments and the window from there
template <typename P>
P* after_sinks(const Shape& s, P* p) {
  const size_t esz = s.dt == RADAR_BF16 ? 2 : 4;
  using B = typename std::conditional<std::is_const<P>::value, const unsigned char,
                                      unsigned char>::type;
  return reinterpret_cast<P*>(reinterpret_cast<B*>(p) + (size_t)s.n_sink * s.d * esz);
}

// ---- decode pieces -------------------------------------------------------
template <typename T, int D, int G>
void launch_phi_q_g(const Shape& s, const void* q, const void* omega, float* phiq,
                    hipStream_t st) {
  const float s1 = kLog2e / std::pow((float)s.d, 0.25f);
  const float s2 = kLog2e / (2.f * std::sqrt((float)s.d));
  const dim3 grid((unsigned)(s.n / 64), (unsigned)(s.B * s.Hkv));
  if constexpr (sizeof(T) == 2) {
    if (s.obf) {
      launch(RADAR_K_PHI_Q, k_phi_q<T, D, G, true>, grid, dim3(256), 0, st,
             reinterpret_cast<const T*>(q), omega, phiq, s.n, s.Hq, s.Hkv, s1, s2,
             1.f / std::sqrt((float)s.n));
      return;
    }
  }
  launch(RADAR_K_PHI_Q, k_phi_q<T, D, G, false>, grid, dim3(256), 0, st,
         reinterpret_cast<const T*>(q), omega, phiq, s.n, s.Hq, s.Hkv, s1, s2,
         1.f / std::sqrt((float)s.n));
}

template <typename T, int D>
void launch_phi_q(const Shape& s, const void* q, const void* omega, float* phiq,
                  hipStream_t st) {
  switch (s.G) {
    case 1: launch_phi_q_g<T, D, 1>(s, q, omega, phiq, st); break;
    case 2: launch_phi_q_g<T, D, 2>(s, q, omega, phiq, st); break;
    case 4: launch_phi_q_g<T, D, 4>(s, q, omega, phiq, st); break;
    default: launch_phi_q_g<T, D, 8>(s, q, omega, phiq, st); break;
  }
}

// n_cand: the largest candidate count of the call (grid size); each
// workgroup reads its sequence's own from sa
template <int N, int G>
void launch_score_ng(const Shape& s, const float* phiq, const float* summ,
                     float* scores, int n_cand, const SeqArgs& sa, hipStream_t st) {
  constexpr int rows_per_wave = 16 * (N <= 256 ? 2 : 1);
  // waves per workgroup: 4 when that still gives two workgroups per CU,
  // else fewer, so that the rows spread over more CUs
  int wpb = 4;
  while (wpb > 1 && ceil_div(n_cand, rows_per_wave * wpb) * s.B * s.Hkv < 2 * num_cu())
    wpb >>= 1;
  const dim3 grid((unsigned)ceil_div(n_cand, rows_per_wave * wpb), (unsigned)(s.B * s.Hkv));
  const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);
  launch(RADAR_K_SCORE, k_score<N, G>, grid, dim3(64 * wpb), 0, st, phiq, summ, scores,
         s.Hq, s.Hkv, sa, s.s_cap, nc_cap);
}

template <int N>
void launch_score_n(const Shape& s, const float* phiq, const float* summ,
                    float* scores, int n_cand, const SeqArgs& sa, hipStream_t st) {
  switch (s.G) {
    case 1: launch_score_ng<N, 1>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 2: launch_score_ng<N, 2>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 4: launch_score_ng<N, 4>(s, phiq, summ, scores, n_cand, sa, st); break;
    default: launch_score_ng<N, 8>(s, phiq, summ, scores, n_cand, sa, st); break;
  }
}

void launch_score(const Shape& s, const float* phiq, const float* summ,
                  float* scores, int n_cand, const SeqArgs& sa, hipStream_t st) {
  switch (s.n) {
    case 64: launch_score_n<64>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 128: launch_score_n<128>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 256: launch_score_n<256>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 512: launch_score_n<512>(s, phiq, summ, scores, n_cand, sa, st); break;
    case 1024: launch_score_n<1024>(s, phiq, summ, scores, n_cand, sa, st); break;
    default: launch_score_n<2048>(s, phiq, summ, scores, n_cand, sa, st); break;
  }
}

// The merge of the partials into the output: fixed_nwg partials per pair
// (the fused kernel's workgroups), or those of the split attention (tpw);
// partials_per_head bounds their count (at most kMaxWg). Above 128 the dims
// are split over D / 32 workgroups per head; otherwise one 256-thread
// workgroup per head (1024 threads measured the same or up to 0.5 us slower).
template <typename T, int D>
void launch_combine(const Shape& s, const float* part, const int* ucnt, void* out,
                    const SeqArgs& sa, const WsLayout& L, int tpw, int fixed_nwg,
                    int partials_per_head, hipStream_t st) {
  if (partials_per_head > 128)
    launch(RADAR_K_COMBINE, k_combine<T, D, 1024, 32, kMaxWg, 16>,
           dim3((unsigned)(s.B * s.Hq), (unsigned)(D / 32)), dim3(1024), 0, st, part,
           ucnt, reinterpret_cast<T*>(out), s.Hq, s.Hkv, s.G, L.tiles_per_seg, sa,
           L.maxwg, tpw, fixed_nwg);
  else
    launch(RADAR_K_COMBINE, k_combine<T, D, 256, D, 128, 0>, dim3((unsigned)(s.B * s.Hq)),
           dim3(256), 0, st, part, ucnt, reinterpret_cast<T*>(out), s.Hq, s.Hkv, s.G,
           L.tiles_per_seg, sa, L.maxwg, tpw, fixed_nwg);
}

template <typename T, int D, int G>
void launch_attend_g(const Shape& s, const void* q, const void* K, const void* V,
                     unsigned char* w, const WsLayout& L, int grid_x, int tpw,
                     const SeqArgs& sa, hipStream_t st) {
  const float qscale = kLog2e / std::sqrt((float)s.d);
  launch(RADAR_K_ATTEND, k_attend<T, D, G>,
         dim3((unsigned)grid_x, (unsigned)(s.B * s.Hkv)), dim3(256), 0, st,
         reinterpret_cast<const T*>(q), reinterpret_cast<const T*>(K),
         reinterpret_cast<const T*>(V), reinterpret_cast<const int*>(w + L.uni),
         reinterpret_cast<const int*>(w + L.ucnt), reinterpret_cast<float*>(w + L.part),
         s.Hq, s.Hkv, s.cap, L.tiles_per_seg, sa, s.per_head, L.umax, L.maxwg, tpw,
         qscale);
}

template <typename T, int D>
void launch_attend_d(const Shape& s, const void* q, const void* K, const void* V,
                     unsigned char* w, const WsLayout& L, int grid_x, int tpw,
                     const SeqArgs& sa, void* out, hipStream_t st) {
  switch (s.G) {
    case 1: launch_attend_g<T, D, 1>(s, q, K, V, w, L, grid_x, tpw, sa, st); break;
    case 2: launch_attend_g<T, D, 2>(s, q, K, V, w, L, grid_x, tpw, sa, st); break;
    case 4: launch_attend_g<T, D, 4>(s, q, K, V, w, L, grid_x, tpw, sa, st); break;
    default: launch_attend_g<T, D, 8>(s, q, K, V, w, L, grid_x, tpw, sa, st); break;
  }
  launch_combine<T, D>(s, reinterpret_cast<const float*>(w + L.part),
                       reinterpret_cast<const int*>(w + L.ucnt), out, sa, L, tpw, 0,
                       grid_x, st);
}

// Tiles beyond the union's segments per (b, kv head), the window's and the
// sinks': exact for one shared length, an upper bound over lengths in
// [1, t_max] for per-sequence lengths (a window never exceeds w + c - 1
// tokens nor the tokens after the sinks).
int64_t extra_tiles(const Shape& s, const SeqArgs& sa) {
  const Span sp = make_span(sa.t_max, sa);
  const int64_t win = sa.lens ? std::min<int64_t>(sp.t, (int64_t)s.w + s.c - 1)
                              : sp.t - sp.ws;
  return ceil_div(win, kTile) + ceil_div(sp.sink, kTile);
}

// Split of the attention work: tiles per wave (tpw) so that the grid still
// holds about eight workgroups per CU (a grid only just above the resident
// count leaves a long tail), but no more (fewer, larger workgroups mean fewer
// partials to merge); and the grid width per (b, kv head) for the largest
// union.
struct AttendGrid {
  int grid_x, tpw;
};

AttendGrid attend_grid(const Shape& s, const WsLayout& L, int u_bound,
                       int64_t extra) {
  const int64_t per_bh = (int64_t)u_bound * L.tiles_per_seg + extra;
  const int64_t tiles = per_bh * s.B * s.Hkv;
  const int64_t tpw = std::min<int64_t>(8, std::max<int64_t>(1, tiles / (4 * 8 * num_cu())));
  return {(int)ceil_div(per_bh, 4 * tpw), (int)tpw};
}

// exact attention over the union in the workspace, then the merge; K and V
// start after the sinks
radar_status launch_attend(const Shape& s, const void* q, const void* K,
                           const void* V, const AttendGrid& ag, const SeqArgs& sa,
                           void* out, unsigned char* w, const WsLayout& L,
                           hipStream_t st) {
  if (s.dt == RADAR_BF16) {
    if (s.d == 64) launch_attend_d<bf16_t, 64>(s, q, K, V, w, L, ag.grid_x, ag.tpw, sa, out, st);
    else launch_attend_d<bf16_t, 128>(s, q, K, V, w, L, ag.grid_x, ag.tpw, sa, out, st);
  } else {
    if (s.d == 64) launch_attend_d<float, 64>(s, q, K, V, w, L, ag.grid_x, ag.tpw, sa, out, st);
    else launch_attend_d<float, 128>(s, q, K, V, w, L, ag.grid_x, ag.tpw, sa, out, st);
  }
  return launch_status();
}

// ---- exact segment search ---------------------------------------------------
template <typename T, int D>
void launch_segment_mass_d(const Shape& s, const void* q, const void* K, float* scores,
                           int n_cand, const SeqArgs& sa, hipStream_t st) {
  const dim3 grid((unsigned)ceil_div(n_cand, 4), (unsigned)(s.B * s.Hkv));
  const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);
  const float qscale = kLog2e / std::sqrt((float)s.d);
  const T* qt = reinterpret_cast<const T*>(q);
  const T* Kt = reinterpret_cast<const T*>(K);
  switch (s.G) {
    case 1: launch(RADAR_K_SCORE, k_segment_mass<T, D, 1>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale); break;
    case 2: launch(RADAR_K_SCORE, k_segment_mass<T, D, 2>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale); break;
    case 4: launch(RADAR_K_SCORE, k_segment_mass<T, D, 4>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale); break;
    default: launch(RADAR_K_SCORE, k_segment_mass<T, D, 8>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale); break;
  }
}

// ---- fused path -------------------------------------------------------------
thread_local int g_path_override = RADAR_PATH_AUTO;

// SEL: the select path (uni_out / ucnt_out / umax receive the union)
template <typename T, int D, int G, int N, bool SEL>
radar_status launch_fused_n(const Shape& s, const void* q, const void* K,
                            const void* V, const void* omega,
                            const float* summ, const SeqArgs& sa, void* out,
                            int32_t* selected, float* sel_scores, int* uni_out,
                            int* ucnt_out, int umax, const AppendArgs& ap,
                            int R, float* part, int maxwg, hipStream_t st) {
  const float s1 = kLog2e / std::pow((float)s.d, 0.25f);
  const float s2 = kLog2e / (2.f * std::sqrt((float)s.d));
  const int n_pairs = s.B * s.Hkv;
  launch(SEL ? RADAR_K_SELECT : RADAR_K_FUSED, k_decode_fused<T, D, G, N, SEL>,
         dim3((unsigned)(n_pairs * R)), dim3(kFusedWaves * 64), 0, st,
         reinterpret_cast<const T*>(q), reinterpret_cast<const T*>(K),
         reinterpret_cast<const T*>(V), omega, s.obf, summ, reinterpret_cast<T*>(out),
         selected, sel_scores, s.Hq, s.Hkv, s.cap, s.s_cap, (int)ceil_div(s.c, kTile),
         sa, s.per_head, s1, s2, 1.f / std::sqrt((float)s.n),
         kLog2e / std::sqrt((float)s.d), uni_out, ucnt_out, umax, ap, R, n_pairs,
         part, maxwg);
  return launch_status();
}

#define RADAR_FUSED_ARGS s, q, K, V, omega, summ, sa, out, selected, sel_scores, uni_out, ucnt_out, umax, ap, R, part, maxwg, st
#define RADAR_FUSED_PARAMS const Shape& s, const void* q, const void* K, const void* V, \
    const void* omega, const float* summ, const SeqArgs& sa, void* out, int32_t* selected, \
    float* sel_scores, int* uni_out, int* ucnt_out, int umax, const AppendArgs& ap, int R, \
    float* part, int maxwg, hipStream_t st

template <typename T, int D, int G, bool SEL>
radar_status launch_fused_g(RADAR_FUSED_PARAMS) {
  switch (s.n) {
    case 64: return launch_fused_n<T, D, G, 64, SEL>(RADAR_FUSED_ARGS);
    case 128: return launch_fused_n<T, D, G, 128, SEL>(RADAR_FUSED_ARGS);
    case 256: return launch_fused_n<T, D, G, 256, SEL>(RADAR_FUSED_ARGS);
    case 512: return launch_fused_n<T, D, G, 512, SEL>(RADAR_FUSED_ARGS);
    case 1024: return launch_fused_n<T, D, G, 1024, SEL>(RADAR_FUSED_ARGS);
    default: return launch_fused_n<T, D, G, 2048, SEL>(RADAR_FUSED_ARGS);
  }
}

template <typename T, int D, bool SEL>
radar_status launch_fused_d(RADAR_FUSED_PARAMS) {
  switch (s.G) {
    case 1: return launch_fused_g<T, D, 1, SEL>(RADAR_FUSED_ARGS);
    case 2: return launch_fused_g<T, D, 2, SEL>(RADAR_FUSED_ARGS);
    default: return launch_fused_g<T, D, 4, SEL>(RADAR_FUSED_ARGS);
  }
}

// K and V start after the sinks. R workgroups per pair; with R > 1 their
// partials go to the workspace and k_combine merges them.
radar_status launch_fused(const Shape& s, const void* q, const void* K, const void* V,
                          const void* omega, const float* summ, const SeqArgs& sa,
                          void* out, int32_t* selected, float* sel_scores,
                          const AppendArgs& ap, int R, unsigned char* w,
                          const WsLayout& L, hipStream_t st) {
  int* uni_out = nullptr;
  int* ucnt_out = nullptr;
  const int umax = 0;
  float* part = R > 1 ? reinterpret_cast<float*>(w + L.part) : nullptr;
  const int maxwg = L.maxwg;
  radar_status r;
  if (s.dt == RADAR_BF16)
    r = s.d == 64 ? launch_fused_d<bf16_t, 64, false>(RADAR_FUSED_ARGS)
                  : launch_fused_d<bf16_t, 128, false>(RADAR_FUSED_ARGS);
  // fp32 caches with d = 128 keep the split path: their tiles need more
  // registers than the fused kernel has to spare
  else if (s.d == 64) r = launch_fused_d<float, 64, false>(RADAR_FUSED_ARGS);
  else return RADAR_EUNSUPPORTED;
  if (r != RADAR_OK || R == 1) return r;
  if (s.dt == RADAR_BF16) {
    if (s.d == 64) launch_combine<bf16_t, 64>(s, part, nullptr, out, sa, L, 1, R, R, st);
    else launch_combine<bf16_t, 128>(s, part, nullptr, out, sa, L, 1, R, R, st);
  } else {
    launch_combine<float, 64>(s, part, nullptr, out, sa, L, 1, R, R, st);
  }
  return launch_status();
}

// the select path's first kernel: phi(q), scores, top-k and union of each
// pair in one workgroup, the union into the workspace
radar_status launch_select(const Shape& s, const void* q, const void* omega,
                           const float* summ, const SeqArgs& sa, int32_t* selected,
                           float* sel_scores, unsigned char* w, const WsLayout& L,
                           const AppendArgs& ap, hipStream_t st) {
  const void* K = nullptr;
  const void* V = nullptr;
  void* out = nullptr;
  int* uni_out = reinterpret_cast<int*>(w + L.uni);
  int* ucnt_out = reinterpret_cast<int*>(w + L.ucnt);
  const int umax = L.umax;
  const int R = 1, maxwg = 0;
  float* part = nullptr;
  if (s.dt == RADAR_BF16)
    return s.d == 64 ? launch_fused_d<bf16_t, 64, true>(RADAR_FUSED_ARGS)
                     : launch_fused_d<bf16_t, 128, true>(RADAR_FUSED_ARGS);
  return s.d == 64 ? launch_fused_d<float, 64, true>(RADAR_FUSED_ARGS)
                   : launch_fused_d<float, 128, true>(RADAR_FUSED_ARGS);
}
#undef RADAR_FUSED_ARGS
#undef RADAR_FUSED_PARAMS

// A pair's HBM bytes in one decode step at length t (summary rows plus the
// K/V of the largest union, the window and the sinks), the quantity one
// fused workgroup streams.
int64_t pair_bytes(const Shape& s, const SeqArgs& sa) {
  const Span sp = make_span(sa.t_max, sa);
  const int64_t u = std::min<int64_t>((int64_t)s.G * sp.k_eff, sp.n_cand);
  const int64_t skv = s.dt == RADAR_BF16 ? 2 : 4;
  return (int64_t)sp.n_cand * s.n * 4 +
         (u * s.c + (sp.t - sp.ws) + sp.sink) * 2 * s.d * skv;
}

// Which decode path a call takes.
//  - fused: the shape fits its LDS plan and either there are enough (b, kv
//    head) pairs to occupy every CU (one workgroup per pair), or each pair's
//    step is small enough (<= 256 KB) that one workgroup streams it in a few
//    microseconds, or a pair's summary rows are few (<= 384 KB): then R
//    workgroups per pair each repeat the selection (the repeated rows mostly
//    hit the caches) and share the attention (measured: 47k vs 36k tokens/s
//    for the select path at 16K, 87k vs 86k at 64K GQA; with the 1.5 MB of
//    rows per pair at 512K the repetition costs more than it saves);
//  - select: fp32 caches with d = 128 (outside the fused kernel's register
//    plan) and summary rows <= 384 KB: one workgroup per pair selects, then
//    the split attention spreads the K/V gather over the chip;
//  - split: phi(q), scores and top-k as separate chip-wide kernels.
int choose_path(const Shape& s, const SeqArgs& sa) {
  const int n_cand = make_span(sa.t_max, sa).n_cand;
  const bool fits_select = s.G <= kFusedMaxG && n_cand <= kFusedMaxCand;
  const bool fits_fused = fits_select && !(s.dt == RADAR_F32 && s.d == 128);
  switch (g_path_override) {
    case RADAR_PATH_SPLIT: return RADAR_PATH_SPLIT;
    case RADAR_PATH_FUSED: return fits_fused ? RADAR_PATH_FUSED : RADAR_PATH_SPLIT;
    case RADAR_PATH_SELECT: return fits_select ? RADAR_PATH_SELECT : RADAR_PATH_SPLIT;
    default: break;
  }
  const bool few_rows = (int64_t)n_cand * s.n * 4 <= (384 << 10);
  if (fits_fused && ((int64_t)s.B * s.Hkv >= num_cu() ||
                     pair_bytes(s, sa) <= (256 << 10) || few_rows))
    return RADAR_PATH_FUSED;
  if (fits_select && few_rows) return RADAR_PATH_SELECT;
  return RADAR_PATH_SPLIT;
}

// Argument checks shared by the decode-side calls: pointers, k, the length
// bound t and the workspace. Fills the per-call sequence arguments.
radar_status check_decode(const radar_config* cfg, Shape* s, int64_t t,
                          const int64_t* lens, int32_t k, void* workspace,
                          size_t workspace_bytes, WsLayout* L, SeqArgs* sa) {
  radar_status r = check_cfg(cfg, s);
  if (r != RADAR_OK) return r;
  if (lens && !aligned16(lens)) return RADAR_EINVAL;
  if (k < 1 || k > kMaxK) return RADAR_EUNSUPPORTED;
  if (t < 1 || t > s->cap) return RADAR_ECAPACITY;
  *L = ws_layout(*s, k);
  if (!workspace || !aligned16(workspace)) return RADAR_EWORKSPACE;
  if (workspace_bytes < L->total) return RADAR_EWORKSPACE;
  *sa = SeqArgs{lens, t, s->c, s->w, s->n_sink, k};
  if (make_span(t, *sa).n_cand > kMaxCand) return RADAR_EUNSUPPORTED;
  return RADAR_OK;
}

// Pointer checks shared by radar_append and radar_append_decode.
radar_status check_append(const radar_config* cfg, Shape* s, const void* K,
                          const void* V, const void* k_new, const void* v_new,
                          const void* omega, const float* summaries,
                          const int64_t* pos) {
  radar_status r = check_cfg(cfg, s);
  if (r != RADAR_OK) return r;
  if (!K || !V || !k_new || !v_new || !omega || !summaries) return RADAR_EINVAL;
  if (!aligned16(K) || !aligned16(V) || !aligned16(k_new) || !aligned16(v_new) ||
      !aligned16(omega) || !aligned16(summaries) || (pos && !aligned16(pos)))
    return RADAR_EINVAL;
  return RADAR_OK;
}

AppendArgs append_args(const Shape& s, void* K, void* V, const void* k_new,
                       const void* v_new, const int64_t* pos, int64_t t) {
  const int esz = s.dt == RADAR_BF16 ? 2 : 4;
  return AppendArgs{static_cast<uint4*>(K), static_cast<uint4*>(V),
                    static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new),
                    pos, t, s.d * esz / 16};
}

// The summary refresh of an append of row t (row pos[b] of sequence b): the
// segment the row completes, if any, with the index build's own code.
radar_status refresh_closed(const Shape& s, const void* K, const void* omega,
                            float* summ, int64_t t, const int64_t* pos,
                            hipStream_t st) {
  const void* Kp = after_sinks(s, K);
  if (pos) return launch_build(s, Kp, omega, summ, 0, 1, pos, st);
  const int64_t row = t - s.n_sink;          // row after the sinks
  if (row >= 0 && (row + 1) % s.c == 0)
    return launch_build(s, Kp, omega, summ, (int)((row + 1) / s.c - 1), 1, nullptr,
                        st);
  return RADAR_OK;
}

// Which kernels a decode runs, decided (and checked) before any launch.
struct DecodePlan {
  int path;
  AttendGrid ag;
  int R;               // fused kernel: workgroups per pair
};

#ifndef RADAR_FUSED_WAYS_MAX
#define RADAR_FUSED_WAYS_MAX 1024
#endif

// Workgroups per pair for the fused kernel: one 512-thread workgroup per
// CU overall, at most one per partial slot of the workspace, and 1 when the
// pairs alone fill the chip or a pair's step is small.
int fused_ways(const Shape& s, const WsLayout& L, const SeqArgs& sa) {
  const int64_t P = (int64_t)s.B * s.Hkv;
  if (P >= num_cu() || pair_bytes(s, sa) <= (256 << 10)) return 1;
  return (int)std::max<int64_t>(
      1, std::min<int64_t>({num_cu() / P, (int64_t)L.maxwg, RADAR_FUSED_WAYS_MAX}));
}

radar_status plan_decode(const Shape& s, const WsLayout& L, const SeqArgs& sa,
                         DecodePlan* p) {
  const Span top = make_span(sa.t_max, sa);
  p->path = choose_path(s, sa);
  p->ag = AttendGrid{0, 1};
  p->R = 1;
  if (p->path == RADAR_PATH_FUSED) {
    p->R = fused_ways(s, L, sa);
    return RADAR_OK;
  }
  const int u_bound = std::min(s.G * top.k_eff, top.n_cand);
  p->ag = attend_grid(s, L, u_bound, extra_tiles(s, sa));
  return p->ag.grid_x > kMaxWg ? RADAR_EUNSUPPORTED : RADAR_OK;
}

// The decode launches. The first per-(b, kv head) kernel of the path (the
// fused kernel, the select kernel or the top-k) also writes the new rows
// that ap describes, before the attention reads them.
radar_status run_decode(const Shape& s, const WsLayout& L, const SeqArgs& sa,
                        const DecodePlan& plan, const void* q, const void* K,
                        const void* V, const void* omega, const float* summaries,
                        void* out, int32_t* selected, float* scores,
                        unsigned char* w, const AppendArgs& ap, hipStream_t stream) {
  const Span top = make_span(sa.t_max, sa);
  const void* Kp = after_sinks(s, K);
  const void* Vp = after_sinks(s, V);
  if (plan.path == RADAR_PATH_FUSED)
    return launch_fused(s, q, Kp, Vp, omega, summaries, sa, out, selected, scores, ap,
                        plan.R, w, L, stream);
  if (plan.path == RADAR_PATH_SELECT) {
    const radar_status r = launch_select(s, q, omega, summaries, sa, selected, scores,
                                         w, L, ap, stream);
    if (r != RADAR_OK) return r;
    return launch_attend(s, q, Kp, Vp, plan.ag, sa, out, w, L, stream);
  }
  float* phiq = reinterpret_cast<float*>(w + L.phiq);
  float* sc = reinterpret_cast<float*>(w + L.scores);
  if (top.n_cand > 0) {
    if (s.dt == RADAR_BF16) {
      if (s.d == 64) launch_phi_q<bf16_t, 64>(s, q, omega, phiq, stream);
      else launch_phi_q<bf16_t, 128>(s, q, omega, phiq, stream);
    } else {
      if (s.d == 64) launch_phi_q<float, 64>(s, q, omega, phiq, stream);
      else launch_phi_q<float, 128>(s, q, omega, phiq, stream);
    }
    launch_score(s, phiq, summaries, sc, top.n_cand, sa, stream);
  }
  launch(RADAR_K_TOPK, k_topk_union, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0, stream,
         sc, s.Hq, s.Hkv, s.G, sa, (int)std::max<int64_t>(1, s.s_cap), s.per_head,
         reinterpret_cast<int*>(w + L.uni), reinterpret_cast<int*>(w + L.ucnt), L.umax,
         selected, scores, ap, s.cap);
  const radar_status r = launch_status();
  if (r != RADAR_OK) return r;
  return launch_attend(s, q, Kp, Vp, plan.ag, sa, out, w, L, stream);
}

radar_status append_decode_impl(const radar_config* cfg, const void* q, void* K, void* V,
                                const void* k_new, const void* v_new, const void* omega,
                                float* summaries, int64_t t, const int64_t* pos,
                                int32_t k, void* out, int32_t* selected, float* scores,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  Shape s;
  radar_status r = check_append(cfg, &s, K, V, k_new, v_new, omega, summaries, pos);
  if (r != RADAR_OK) return r;
  if (!q || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(out) || (selected && !aligned16(selected)) ||
      (scores && !aligned16(scores)))
    return RADAR_EINVAL;
  WsLayout L;
  SeqArgs sa;
  r = check_decode(cfg, &s, t, pos, k, workspace, workspace_bytes, &L, &sa);
  if (r != RADAR_OK) return r;
  sa.lens_add = pos ? 1 : 0;
  DecodePlan plan;
  r = plan_decode(s, L, sa, &plan);
  if (r != RADAR_OK) return r;
  unsigned char* w = static_cast<unsigned char*>(workspace);
  const AppendArgs ap = append_args(s, K, V, k_new, v_new, pos, t - 1);
  if (s.w == 0) {
    // Without a window the segment this row completes is already a
    // candidate of the same step: write the row and refresh its summary
    // first, then decode.
    launch(RADAR_K_APPEND, k_append, dim3((unsigned)(s.B * s.Hkv)), dim3(64), 0,
           stream, ap, s.cap, s.Hkv);
    r = launch_status();
    if (r == RADAR_OK) r = refresh_closed(s, K, omega, summaries, t - 1, pos, stream);
    if (r != RADAR_OK) return r;
    return run_decode(s, L, sa, plan, q, K, V, omega, summaries, out, selected, scores,
                      w, AppendArgs{}, stream);
  }
  // With w >= 1 the completed segment ends inside the window, so the decode
  // does not read its summary: the refresh runs after it.
  r = run_decode(s, L, sa, plan, q, K, V, omega, summaries, out, selected, scores, w,
                 ap, stream);
  if (r != RADAR_OK) return r;
  return refresh_closed(s, K, omega, summaries, t - 1, pos, stream);
}


// ---- the decode scratch without allocation ---------------------------------
// radar_append_decode_noalloc keeps the decode's workspace in this array
// instead of a caller buffer: one copy per GPU the library runs on (the
// loader places it with the code object), held until the process ends.
// Host code never passes the array's name to a kernel (on the host it is
// only a stand-in for the symbol): the device address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
constexpr size_t kScratchBytes = RADAR_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch address on the device of `stream` (which must be the current
// device: the lookup runs with it current).
radar_status scratch_of(hipStream_t stream, void** out) {
  int cur = -1, dev = -1;
  if (hipGetDevice(&cur) != hipSuccess) return launch_status();
  if (stream) {
    if (hipStreamGetDevice(stream, &dev) != hipSuccess) return launch_status();
  } else {
    dev = cur;
  }
  if (dev != cur) return RADAR_EINVAL;
  if (dev < 0 || dev >= kMaxDevices) return RADAR_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      snprintf(g_last_error, sizeof g_last_error, "hipGetSymbolAddress: %s",
               hipGetErrorString(e));
      (void)hipGetLastError();
      return RADAR_EHIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RADAR_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

int32_t radar_abi_version(void) { return RADAR_ABI_VERSION; }

radar_status radar_schedule_sqrt(int64_t t, int32_t* seg_len, int32_t* window) {
  if (!seg_len || !window) return RADAR_EINVAL;
  if (t < 1 || t > ((int64_t)1 << 31)) return RADAR_ECAPACITY;
  int64_t c = (int64_t)std::sqrt((double)t);
  while (c * c > t) --c;
  while ((c + 1) * (c + 1) <= t) ++c;
  *seg_len = (int32_t)c;
  *window = (int32_t)(t - c * c);
  return RADAR_OK;
}

radar_status radar_set_decode_path(int32_t path) {
  if (path != RADAR_PATH_AUTO && path != RADAR_PATH_SPLIT && path != RADAR_PATH_FUSED &&
      path != RADAR_PATH_SELECT)
    return RADAR_EINVAL;
  g_path_override = path;
  return RADAR_OK;
}

int32_t radar_decode_path(const radar_config* cfg, int64_t t, int32_t k) {
  Shape s;
  if (check_cfg(cfg, &s) != RADAR_OK || k < 1 || k > kMaxK || t < 1 || t > s.cap)
    return -1;
  return choose_path(s, SeqArgs{nullptr, t, s.c, s.w, s.n_sink, k});
}

radar_status radar_profile_enable(int32_t on) {
  g_prof.on = on != 0;
  return RADAR_OK;
}

size_t radar_peak_sink_floats(void) {
  return (size_t)num_cu() * kPeakWgPerCu * 256;
}

radar_status radar_peak_mfma(int32_t iters, float* sink, double* work,
                             hipStream_t stream) {
  if (iters < 1 || !sink || !work || !aligned16(sink)) return RADAR_EINVAL;
  const unsigned grid = (unsigned)(num_cu() * kPeakWgPerCu);
  hipLaunchKernelGGL(k_peak_mfma, dim3(grid), dim3(256), 0, stream, iters, sink);
  *work = (double)grid * 4 * iters * 8 * (2.0 * 16 * 16 * 32);
  return launch_status();
}

radar_status radar_peak_exp(int32_t iters, float* sink, double* work,
                            hipStream_t stream) {
  if (iters < 1 || !sink || !work || !aligned16(sink)) return RADAR_EINVAL;
  const unsigned grid = (unsigned)(num_cu() * kPeakWgPerCu);
  hipLaunchKernelGGL(k_peak_exp, dim3(grid), dim3(256), 0, stream, iters, sink);
  *work = (double)grid * 256 * iters * 8;
  return launch_status();
}

radar_status radar_profile_read(double* ms, int64_t* launches, int32_t n) {
  if (!ms || !launches || n < RADAR_K_COUNT) return RADAR_EINVAL;
  for (int i = 0; i < n; ++i) { ms[i] = 0.0; launches[i] = 0; }
  radar_status st = RADAR_OK;
  for (const auto& r : g_prof.recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess ||
        hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) {
      snprintf(g_last_error, sizeof g_last_error, "%s",
               hipGetErrorString(hipGetLastError()));
      st = RADAR_EHIP;
    } else {
      ms[r.kind] += t;
      launches[r.kind] += 1;
    }
    g_prof.pool.push_back(r.a);
    g_prof.pool.push_back(r.b);
  }
  g_prof.recs.clear();
  return st;
}

const char* radar_last_error(void) { return g_last_error; }

const char* radar_status_string(radar_status st) {
  switch (st) {
    case RADAR_OK: return "ok";
    case RADAR_EINVAL: return "invalid argument";
    case RADAR_ECAPACITY: return "position outside the cache capacity";
    case RADAR_EUNSUPPORTED: return "shape outside the instantiated kernels";
    case RADAR_EHIP: return "HIP launch failed";
    case RADAR_EWORKSPACE: return "workspace missing or too small";
  }
  return "unknown status";
}

size_t radar_decode_workspace_bytes(const radar_config* cfg, int32_t k) {
  Shape s;
  if (check_cfg(cfg, &s) != RADAR_OK || k < 1 || k > kMaxK) return 0;
  return ws_layout(s, k).total;
}

radar_status radar_build_index(const radar_config* cfg, const void* K,
                               const void* omega, int64_t t, float* summaries,
                               hipStream_t stream) {
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (!K || !omega || !summaries) return RADAR_EINVAL;
  if (!aligned16(K) || !aligned16(omega) || !aligned16(summaries)) return RADAR_EINVAL;
  if (t < 1 || t > s.cap) return RADAR_ECAPACITY;
  const int64_t n_seg = std::max<int64_t>(0, t - s.n_sink) / s.c;
  if (n_seg == 0) return RADAR_OK;
  return launch_build(s, after_sinks(s, K), omega, summaries, 0, (int)n_seg,
                      nullptr, stream);
}

radar_status radar_append(const radar_config* cfg, void* K, void* V,
                          const void* k_new, const void* v_new,
                          const void* omega, int64_t t, const int64_t* pos,
                          float* summaries, hipStream_t stream) {
  Shape s;
  radar_status r = check_append(cfg, &s, K, V, k_new, v_new, omega, summaries, pos);
  if (r != RADAR_OK) return r;
  if (!pos && (t < 0 || t >= s.cap)) return RADAR_ECAPACITY;
  const AppendArgs ap = append_args(s, K, V, k_new, v_new, pos, t);
  launch(RADAR_K_APPEND, k_append, dim3((unsigned)(s.B * s.Hkv)), dim3(64), 0, stream,
         ap, s.cap, s.Hkv);
  r = launch_status();
  if (r != RADAR_OK) return r;
  return refresh_closed(s, K, omega, summaries, t, pos, stream);
}

radar_status radar_decode(const radar_config* cfg, const void* q, const void* K,
                          const void* V, const void* omega,
                          const float* summaries, int64_t t, const int64_t* lens,
                          int32_t k, void* out, int32_t* selected, float* scores,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (!cfg || !q || !K || !V || !omega || !summaries || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(omega) ||
      !aligned16(summaries) || !aligned16(out) ||
      (selected && !aligned16(selected)) || (scores && !aligned16(scores)))
    return RADAR_EINVAL;
  Shape s;
  WsLayout L;
  SeqArgs sa;
  radar_status r = check_decode(cfg, &s, t, lens, k, workspace, workspace_bytes, &L, &sa);
  if (r != RADAR_OK) return r;
  DecodePlan plan;
  r = plan_decode(s, L, sa, &plan);
  if (r != RADAR_OK) return r;
  return run_decode(s, L, sa, plan, q, K, V, omega, summaries, out, selected, scores,
                    static_cast<unsigned char*>(workspace), AppendArgs{}, stream);
}

radar_status radar_append_decode(const radar_config* cfg, const void* q, void* K,
                                 void* V, const void* k_new, const void* v_new,
                                 const void* omega, float* summaries, int64_t t,
                                 const int64_t* pos, int32_t k, void* out,
                                 int32_t* selected, float* scores, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  return append_decode_impl(cfg, q, K, V, k_new, v_new, omega, summaries, t, pos, k,
                            out, selected, scores, workspace, workspace_bytes, stream);
}

radar_status radar_append_decode_noalloc(const radar_config* cfg, const void* q,
                                         void* K, void* V, const void* k_new,
                                         const void* v_new, const void* omega,
                                         float* summaries, int64_t t,
                                         const int64_t* pos, int32_t k, void* out,
                                         int32_t* selected, float* scores,
                                         hipStream_t stream) {
  Shape s;
  if (check_cfg(cfg, &s) != RADAR_OK || k < 1 || k > kMaxK)
    return append_decode_impl(cfg, q, K, V, k_new, v_new, omega, summaries, t, pos, k,
                              out, selected, scores, nullptr, 0, stream);
  if (ws_layout(s, k).total > kScratchBytes) return RADAR_EWORKSPACE;
  void* w = nullptr;
  const radar_status r = scratch_of(stream, &w);
  if (r != RADAR_OK) return r;
  return append_decode_impl(cfg, q, K, V, k_new, v_new, omega, summaries, t, pos, k,
                            out, selected, scores, w, kScratchBytes, stream);
}


radar_status radar_decode_exact(const radar_config* cfg, const void* q,
                                const void* K, const void* V, int64_t t,
                                const int64_t* lens, int32_t k, void* out,
                                int32_t* selected, float* scores,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  if (!cfg || !q || !K || !V || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(out) ||
      (selected && !aligned16(selected)) || (scores && !aligned16(scores)))
    return RADAR_EINVAL;
  Shape s;
  WsLayout L;
  SeqArgs sa;
  radar_status r = check_decode(cfg, &s, t, lens, k, workspace, workspace_bytes, &L, &sa);
  if (r != RADAR_OK) return r;
  const Span top = make_span(t, sa);
  const void* Kp = after_sinks(s, K);
  const void* Vp = after_sinks(s, V);
  const int u_bound = std::min(s.G * top.k_eff, top.n_cand);
  const AttendGrid ag = attend_grid(s, L, u_bound, extra_tiles(s, sa));
  if (ag.grid_x > kMaxWg) return RADAR_EUNSUPPORTED;

  unsigned char* w = reinterpret_cast<unsigned char*>(workspace);
  float* sc = reinterpret_cast<float*>(w + L.scores);
  if (top.n_cand > 0) {
    if (s.dt == RADAR_BF16) {
      if (s.d == 64) launch_segment_mass_d<bf16_t, 64>(s, q, Kp, sc, top.n_cand, sa, stream);
      else launch_segment_mass_d<bf16_t, 128>(s, q, Kp, sc, top.n_cand, sa, stream);
    } else {
      if (s.d == 64) launch_segment_mass_d<float, 64>(s, q, Kp, sc, top.n_cand, sa, stream);
      else launch_segment_mass_d<float, 128>(s, q, Kp, sc, top.n_cand, sa, stream);
    }
  }
  launch(RADAR_K_TOPK, k_topk_union, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0, stream,
         sc, s.Hq, s.Hkv, s.G, sa, (int)std::max<int64_t>(1, s.s_cap), s.per_head,
         reinterpret_cast<int*>(w + L.uni), reinterpret_cast<int*>(w + L.ucnt), L.umax,
         selected, scores, AppendArgs{}, s.cap);
  r = launch_status();
  if (r != RADAR_OK) return r;
  return launch_attend(s, q, Kp, Vp, ag, sa, out, w, L, stream);
}

radar_status radar_attend_selected(const radar_config* cfg, const void* q,
                                   const void* K, const void* V,
                                   const int32_t* selected, int32_t k, int64_t t,
                                   const int64_t* lens, void* out,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  if (!cfg || !q || !K || !V || !selected || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(selected) ||
      !aligned16(out))
    return RADAR_EINVAL;
  Shape s;
  WsLayout L;
  SeqArgs sa;
  radar_status r = check_decode(cfg, &s, t, lens, k, workspace, workspace_bytes, &L, &sa);
  if (r != RADAR_OK) return r;
  const Span top = make_span(t, sa);
  const int u_bound = std::min(s.G * k, top.n_cand);
  const AttendGrid ag = attend_grid(s, L, u_bound, extra_tiles(s, sa));
  if (ag.grid_x > kMaxWg) return RADAR_EUNSUPPORTED;
  unsigned char* w = reinterpret_cast<unsigned char*>(workspace);
  launch(RADAR_K_TOPK, k_union_given, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0,
         stream, selected, k, s.Hq, s.Hkv, s.G, sa, s.per_head,
         reinterpret_cast<int*>(w + L.uni), reinterpret_cast<int*>(w + L.ucnt),
         L.umax);
  r = launch_status();
  if (r != RADAR_OK) return r;
  return launch_attend(s, q, after_sinks(s, K), after_sinks(s, V), ag, sa, out, w,
                       L, stream);
}

}  // extern "C"

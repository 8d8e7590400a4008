// Radar decode path on MI355X (gfx950, CDNA4): kernels and the C ABI.
//
// Kernels (one launch each, all on the caller's stream):
//   k_build       segment summaries, Eq. 4 + Eq. 5: bf16/fp32 matrix-core
//                 projection of the keys onto Omega, exp2 epilogue, mean over
//                 the segment's tokens. Also serves the segment close of
//                 radar_append, so appends and rebuilds agree bit for bit.
//   k_append      writes one k/v row per (b, kv head).
//   k_phi_q       phi(q) of every query head, Eq. 4.
//   k_score       Eq. 6 scores of every candidate segment: HBM-bound GEMV
//                 over the fp32 summaries, cross-lane transpose-reduce.
//   k_topk_union  per query head top-k (score desc, index asc) by wavefront
//                 arg-max rounds; per kv head sorted union of the group.
//   k_attend      exact attention (Eq. 1-2) over the union's segments plus
//                 the window: coalesced 16-byte gathers of K/V, fp32 online
//                 softmax, one partial (max, sum, acc[d]) per workgroup.
//   k_combine     log-sum-exp merge of the partials into the output.
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
#include <vector>

#include "radar.h"

namespace {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr int kWave = 64;
constexpr int kTile = 64;          // tokens per wave in k_attend / k_build
constexpr int kMaxK = 256;         // largest k accepted
constexpr int kMaxG = 8;           // largest query-head group
constexpr int kMaxCand = 2048;     // largest number of candidate segments

typedef uint16_t bf16_t;           // storage type of a bfloat16 value
typedef unsigned long long u64;   // 64-bit type of the wave shuffles
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

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

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN)
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u)
    return (u >> 16) | ((u & 0xffffu) ? 0x40u : 0u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
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

// One step of a cross-lane transpose-reduce: NV values per lane, lanes that
// differ in bit MASK exchange half of them, so afterwards v[0 .. NV/2) hold
// pair sums and the upper/lower half kept is selected by (lane & MASK).
template <int NV, int MASK>
__device__ __forceinline__ void halve(float* v, int lane) {
  const bool up = (lane & MASK) != 0;
#pragma unroll
  for (int i = 0; i < NV / 2; ++i) {
    const float keep = up ? v[i + NV / 2] : v[i];
    const float send = up ? v[i] : v[i + NV / 2];
    v[i] = keep + __shfl_xor(send, MASK);
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmaxf(v, __shfl_xor(v, m));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m);
  return v;
}

// ---------------------------------------------------------------------------
// k_build: segment summaries (Eq. 4, Eq. 5)
// ---------------------------------------------------------------------------
// Work item = one (b, kv head, segment) and one slice of 64*FT features.
// Wave w of the workgroup owns features [w*16*FT, (w+1)*16*FT) of the slice
// and keeps that slice of Omega (rounded to the MFMA input type) resident in
// registers as MFMA B operands for the whole kernel. Keys stream through LDS
// in tiles of 64 tokens (register-prefetched one tile ahead); every wave
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
    const T* __restrict__ K, const float* __restrict__ omega,
    float* __restrict__ summ, int n, int c, int64_t cap, int64_t s_cap,
    int seg_first, int seg_count, int64_t n_items, float s1, float s2,
    float out_scale, int64_t kv_head_stride_rows) {
  using MC = MfmaCfg<T>;
  using BT = BuildTile<T, D>;
  constexpr int KB = D / MC::kK;
  constexpr int CPR = BT::kChunksPerRow;
  constexpr int CPT = BT::kChunksPerThread;
  static_assert(CPT >= 1 && (256 % CPR) == 0, "tile shape");

  __shared__ __attribute__((aligned(16))) unsigned char tile_lds[kTile * BT::kPitch];
  __shared__ float nrm_lds[kTile];

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
    const float* orow = omega + (int64_t)(fbase + f * 16 + col) * D;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if constexpr (sizeof(T) == 2) {
        const float4 a = *reinterpret_cast<const float4*>(orow + kb * 32 + grp * 8);
        const float4 b = *reinterpret_cast<const float4*>(orow + kb * 32 + grp * 8 + 4);
        bf16x8_t v;
        v[0] = (short)f32_to_bf16(a.x); v[1] = (short)f32_to_bf16(a.y);
        v[2] = (short)f32_to_bf16(a.z); v[3] = (short)f32_to_bf16(a.w);
        v[4] = (short)f32_to_bf16(b.x); v[5] = (short)f32_to_bf16(b.y);
        v[6] = (short)f32_to_bf16(b.z); v[7] = (short)f32_to_bf16(b.w);
        bfrag[f][kb] = v;
      } else {
        bfrag[f][kb] = orow[kb * 4 + grp];
      }
    }
  }

  const int ntiles = (c + kTile - 1) / kTile;
  float psum[FT];
#pragma unroll
  for (int f = 0; f < FT; ++f) psum[f] = 0.f;

  // address of tile `tl` of item `it`
  auto tile_src = [&](int64_t it, int tl, int& valid) -> const T* {
    const int64_t bh = it / seg_count;
    const int64_t s = seg_first + (it % seg_count);
    const int64_t row0 = s * (int64_t)c + (int64_t)tl * kTile;
    valid = min(kTile, c - tl * kTile);
    return K + bh * kv_head_stride_rows * D + row0 * D;
  };

  uint4 pre[CPT];
  int pre_valid = 0;
  int64_t item = blockIdx.x;
  int tl = 0;
  auto fetch = [&](int64_t it, int t_) {
    const T* src = tile_src(it, t_, pre_valid);
#pragma unroll
    for (int p = 0; p < CPT; ++p) {
      const int ci = p * 256 + tid;
      const int row = ci / CPR, ch = ci % CPR;
      if (row < pre_valid)
        pre[p] = *reinterpret_cast<const uint4*>(
            reinterpret_cast<const unsigned char*>(src + (int64_t)row * D) + ch * 16);
      else
        pre[p] = make_uint4(0u, 0u, 0u, 0u);
    }
  };
  if (item < n_items) fetch(item, 0);

  while (item < n_items) {
    const int valid = pre_valid;
    __syncthreads();                       // previous tile fully consumed
#pragma unroll
    for (int p = 0; p < CPT; ++p) {
      const int ci = p * 256 + tid;
      const int row = ci / CPR, ch = ci % CPR;
      *reinterpret_cast<uint4*>(tile_lds + row * BT::kPitch + ch * 16) = pre[p];
      float e[16 / sizeof(T)];
      unpack16<T>(pre[p], e);
      float sq = 0.f;
#pragma unroll
      for (int i = 0; i < (int)(16 / sizeof(T)); ++i) sq = fmaf(e[i], e[i], sq);
#pragma unroll
      for (int m = 1; m < CPR; m <<= 1) sq += __shfl_xor(sq, m);
      if (ch == 0) nrm_lds[row] = sq * s2;
    }
    __syncthreads();

    // prefetch the next tile while this one is multiplied
    int64_t nitem = item;
    int ntl = tl + 1;
    if (ntl == ntiles) { nitem += gridDim.x; ntl = 0; }
    if (nitem < n_items) fetch(nitem, ntl);

#pragma unroll
    for (int st = 0; st < kTile / 16; ++st) {
      if (st * 16 >= valid) break;
      typename MC::frag_t afrag[KB];
      const unsigned char* arow = tile_lds + (st * 16 + col) * BT::kPitch;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        if constexpr (sizeof(T) == 2)
          afrag[kb] = *reinterpret_cast<const bf16x8_t*>(arow + (kb * 32 + grp * 8) * 2);
        else
          afrag[kb] = *reinterpret_cast<const float*>(arow + (kb * 4 + grp) * 4);
      }
      float nb[4];
      bool ok[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = st * 16 + grp * 4 + j;
        nb[j] = nrm_lds[r];
        ok[j] = r < valid;
      }
#pragma unroll
      for (int f = 0; f < FT; ++f) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          if constexpr (sizeof(T) == 2)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[kb], bfrag[f][kb], acc, 0, 0, 0);
          else
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(afrag[kb], bfrag[f][kb], acc, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float v = fast_exp2(fmaf(acc[j], s1, -nb[j]));
          psum[f] += ok[j] ? v : 0.f;
        }
      }
    }

    if (tl == ntiles - 1) {                // segment complete
      const int64_t bh = item / seg_count;
      const int64_t s = seg_first + (item % seg_count);
      float* dst = summ + (bh * s_cap + s) * n + fbase;
#pragma unroll
      for (int f = 0; f < FT; ++f) {
        float v = psum[f];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (lane < 16) dst[f * 16 + col] = v * out_scale;
        psum[f] = 0.f;
      }
    }
    item = nitem;
    tl = ntl;
  }
}

// ---------------------------------------------------------------------------
// k_append: K[b][h][t] = k_new[b][h], V likewise
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(64) void k_append(T* __restrict__ K, T* __restrict__ V,
                                               const T* __restrict__ kn,
                                               const T* __restrict__ vn,
                                               int64_t cap, int64_t t) {
  constexpr int CPR = D * (int)sizeof(T) / 16;
  const int64_t bh = blockIdx.x;
  const int i = threadIdx.x;
  if (i < CPR) {
    const uint4* sk = reinterpret_cast<const uint4*>(kn + bh * D) + i;
    const uint4* sv = reinterpret_cast<const uint4*>(vn + bh * D) + i;
    uint4* dk = reinterpret_cast<uint4*>(K + (bh * cap + t) * D) + i;
    uint4* dv = reinterpret_cast<uint4*>(V + (bh * cap + t) * D) + i;
    *dk = *sk;
    *dv = *sv;
  }
}

// ---------------------------------------------------------------------------
// k_phi_q: phi(q) for every (b, q head), Eq. 4
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void k_phi_q(const T* __restrict__ q,
                                               const float* __restrict__ omega,
                                               float* __restrict__ phiq, int n,
                                               float s1, float s2,
                                               float inv_sqrt_n) {
  __shared__ float qf[D];
  const int64_t bhq = blockIdx.x;
  const int tid = threadIdx.x;
  if (tid < D) qf[tid] = to_f32<T>(q[bhq * D + tid]);
  __syncthreads();
  float nrm = 0.f;
#pragma unroll 8
  for (int e = 0; e < D; ++e) nrm = fmaf(qf[e], qf[e], nrm);
  for (int f = tid; f < n; f += 256) {
    const float4* orow = reinterpret_cast<const float4*>(omega + (int64_t)f * D);
    float dot = 0.f;
#pragma unroll 4
    for (int e4 = 0; e4 < D / 4; ++e4) {
      float4 o = orow[e4];
      if constexpr (sizeof(T) == 2) {
        o.x = round_bf16(o.x); o.y = round_bf16(o.y);
        o.z = round_bf16(o.z); o.w = round_bf16(o.w);
      }
      dot = fmaf(o.x, qf[4 * e4 + 0], dot);
      dot = fmaf(o.y, qf[4 * e4 + 1], dot);
      dot = fmaf(o.z, qf[4 * e4 + 2], dot);
      dot = fmaf(o.w, qf[4 * e4 + 3], dot);
    }
    phiq[bhq * n + f] = fast_exp2(fmaf(dot, s1, -nrm * s2)) * inv_sqrt_n;
  }
}

// ---------------------------------------------------------------------------
// k_score: a[h][s] = phi(q_h) . summ[s], Eq. 6
// ---------------------------------------------------------------------------
// Workgroup = 4 waves x 16 rows. Lane l holds features [l*FPL, (l+1)*FPL) of
// phi(q) for the G heads of the group; each summary row is read as one
// contiguous n*4-byte wave load, and 16 rows' partial dots are reduced across
// the wave by a transpose-reduce (17 shuffles per 16 rows).
template <int N, int G>
__global__ __launch_bounds__(256) void k_score(const float* __restrict__ phiq,
                                               const float* __restrict__ summ,
                                               float* __restrict__ scores,
                                               int Hq, int Hkv, int n_cand,
                                               int64_t s_cap, int nc_cap) {
  constexpr int FPL = N / 64;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int row0 = blockIdx.x * 64 + wave * 16;
  if (row0 >= n_cand) return;

  float pq[G][FPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float* src = phiq + ((b * Hq + hk * G + g) * N) + lane * FPL;
#pragma unroll
    for (int e = 0; e < FPL; ++e) pq[g][e] = src[e];
  }
  float part[G][16];
  const float* base = summ + (bh * s_cap) * N + lane * FPL;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = row0 + r;
    float x[FPL];
    if (row < n_cand) {
      const float* src = base + (int64_t)row * N;
      if constexpr (FPL % 4 == 0) {
#pragma unroll
        for (int e = 0; e < FPL; e += 4) {
          const float4 v = *reinterpret_cast<const float4*>(src + e);
          x[e] = v.x; x[e + 1] = v.y; x[e + 2] = v.z; x[e + 3] = v.w;
        }
      } else if constexpr (FPL == 2) {
        const float2 v = *reinterpret_cast<const float2*>(src);
        x[0] = v.x; x[1] = v.y;
      } else {
        x[0] = src[0];
      }
    } else {
#pragma unroll
      for (int e = 0; e < FPL; ++e) x[e] = 0.f;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < FPL; ++e) acc = fmaf(x[e], pq[g][e], acc);
      part[g][r] = acc;
    }
  }
  const int row = row0 + ((lane >> 2) & 15);
#pragma unroll
  for (int g = 0; g < G; ++g) {
    halve<16, 32>(part[g], lane);
    halve<8, 16>(part[g], lane);
    halve<4, 8>(part[g], lane);
    halve<2, 4>(part[g], lane);
    float v = part[g][0];
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 1);
    if ((lane & 3) == 0 && row < n_cand)
      scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + row] = v;
  }
}

// ---------------------------------------------------------------------------
// k_topk_union: per-head top-k and per-kv-head union
// ---------------------------------------------------------------------------
// Order key of (score, index): larger key = better; ties in score go to the
// lower segment index. Keys are unique because indices are.
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
__device__ __forceinline__ u64 wave_max_u64(u64 v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    const u64 o = __shfl_xor(v, m);
    v = o > v ? o : v;
  }
  return v;
}

// Union of the group's selections: sel[0 .. M) holds segment ids (-1 = none);
// writes the distinct ids in ascending order to uni and their count to *ucnt.
__device__ void group_union(const int* sel, unsigned char* first, int M,
                            int* uni, int* ucnt, int* cnt_lds) {
  const int tid = threadIdx.x;
  if (tid == 0) *cnt_lds = 0;
  for (int i = tid; i < M; i += blockDim.x) {
    const int id = sel[i];
    bool f = id >= 0;
    for (int j = 0; j < i && f; ++j) f = sel[j] != id;
    first[i] = f;
  }
  __syncthreads();
  int mine = 0;
  for (int i = tid; i < M; i += blockDim.x) {
    if (!first[i]) continue;
    const int id = sel[i];
    int rank = 0;
    for (int j = 0; j < M; ++j) rank += (first[j] && sel[j] < id) ? 1 : 0;
    uni[rank] = id;
    ++mine;
  }
  if (mine) atomicAdd(cnt_lds, mine);
  __syncthreads();
  if (tid == 0) *ucnt = *cnt_lds;
}

__global__ __launch_bounds__(256) void k_topk_union(
    const float* __restrict__ scores, int Hq, int Hkv, int G, int n_cand,
    int nc_cap, int k, int k_eff, int* __restrict__ uni,
    int* __restrict__ ucnt, int umax, int32_t* __restrict__ selected,
    float* __restrict__ sel_scores, const int32_t* __restrict__ given,
    int given_k) {
  extern __shared__ float sc_lds[];          // [4 waves][npl][64]
  __shared__ int sel_lds[kMaxG * kMaxK];
  __shared__ unsigned char first_lds[kMaxG * kMaxK];
  __shared__ int cnt_lds;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t bh = blockIdx.x;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  int M;

  if (given == nullptr) {
    const int npl = (n_cand + 63) / 64;
    float* mine = sc_lds + wave * npl * 64;
    for (int hl = wave; hl < G; hl += 4) {
      const int64_t hq = hk * G + hl;
      const float* src = scores + (b * Hq + hq) * (int64_t)nc_cap;
      // each lane keeps the scores of segments lane, lane+64, ... in its own
      // LDS column (only the owning lane ever reads them back)
      u64 best = 0;
      for (int m = 0; m < npl; ++m) {
        const int idx = m * 64 + lane;
        const float v = idx < n_cand ? src[idx] : 0.f;
        mine[m * 64 + lane] = v;
        if (idx < n_cand) {
          const u64 key = order_key(v, idx);
          best = key > best ? key : best;
        }
      }
      int32_t* sel_out = selected ? selected + (b * Hq + hq) * (int64_t)k : nullptr;
      float* sc_out = sel_scores ? sel_scores + (b * Hq + hq) * (int64_t)k : nullptr;
      for (int r = 0; r < k_eff; ++r) {
        const u64 win = wave_max_u64(best);
        const int idx = key_index(win);
        if (lane == 0) {
          sel_lds[hl * k_eff + r] = idx;
          if (sel_out) sel_out[r] = idx;
          if (sc_out) sc_out[r] = key_score(win);
        }
        if ((idx & 63) == lane) {            // owner: next best below `win`
          best = 0;
          for (int m = 0; m < npl; ++m) {
            const int j = m * 64 + lane;
            if (j < n_cand) {
              const u64 key = order_key(mine[m * 64 + lane], j);
              if (key < win && key > best) best = key;
            }
          }
        }
      }
      for (int r = k_eff + lane; r < k; r += 64) {
        if (sel_out) sel_out[r] = -1;
        if (sc_out) sc_out[r] = __uint_as_float(0x7fc00000u);
      }
    }
    M = G * k_eff;
  } else {
    M = G * given_k;
    for (int i = tid; i < M; i += 256) {
      const int hl = i / given_k, r = i % given_k;
      const int id = given[(b * Hq + hk * G + hl) * (int64_t)given_k + r];
      sel_lds[i] = (id >= 0 && id < n_cand) ? id : -1;
    }
  }
  __syncthreads();
  group_union(sel_lds, first_lds, M, uni + bh * umax, ucnt + bh, &cnt_lds);
}

// ---------------------------------------------------------------------------
// k_attend: exact attention over union segments + window, one partial per WG
// ---------------------------------------------------------------------------
// The attended tokens of a (b, kv head) are cut into tiles of <= 64 tokens
// that never cross a segment or the window boundary: tiles_per_seg tiles per
// union segment, then ceil(|W| / 64) window tiles. Workgroup j takes tiles
// 4j .. 4j+3, one per wave. In a wave, lane (r, jj) (r = lane / LPR) reads
// the 16-byte chunk jj of rows r, r + RPI, ... so every load instruction
// covers RPI whole rows contiguously; q.k partials are transpose-reduced so
// that each lane ends with one token's logit, softmax runs across the wave,
// and p is broadcast back to the lanes that hold the matching V chunks.
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void k_attend(
    const T* __restrict__ q, const T* __restrict__ K, const T* __restrict__ V,
    const int* __restrict__ uni, const int* __restrict__ ucnt,
    float* __restrict__ part, int Hq, int Hkv, int64_t cap, int c,
    int tiles_per_seg, int64_t ws, int64_t t, int umax, int maxwg,
    float qscale) {
  constexpr int EPL = Elem<T>::kPer16;     // elements per 16-byte chunk
  constexpr int LPR = D / EPL;             // lanes per row
  constexpr int RPI = kWave / LPR;         // rows per load instruction
  constexpr int ITER = kTile / RPI;        // load instructions per tile
  static_assert(ITER == LPR, "tile shape");
  constexpr int PSTRIDE = D + 4;

  __shared__ float wm[4][G], wl[4][G];
  __shared__ __attribute__((aligned(16))) float wacc[4][G][D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int j = blockIdx.x;

  const int U = ucnt[bh];
  const int seg_tiles = U * tiles_per_seg;
  const int win_tiles = (int)((t - ws + kTile - 1) / kTile);
  const int total = seg_tiles + win_tiles;
  if (j * 4 >= total) return;

  const int ti = j * 4 + wave;
  int64_t start = 0;
  int len = 0;
  if (ti < seg_tiles) {
    const int s = uni[bh * umax + ti / tiles_per_seg];
    const int off = (ti % tiles_per_seg) * kTile;
    start = (int64_t)s * c + off;
    len = min(kTile, c - off);
  } else if (ti < total) {
    start = ws + (int64_t)(ti - seg_tiles) * kTile;
    len = (int)min((int64_t)kTile, t - start);
  }

  const int r = lane / LPR;
  const int jj = lane % LPR;

  float qf[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 u = *reinterpret_cast<const uint4*>(
        q + ((b * Hq + hk * G + g) * D + jj * EPL));
    unpack16<T>(u, qf[g]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[g][e] *= qscale;
  }

  const T* kbase = K + (bh * cap + start) * D + jj * EPL;
  const T* vbase = V + (bh * cap + start) * D + jj * EPL;
  uint4 kr[ITER], vr[ITER];
#pragma unroll
  for (int i = 0; i < ITER; ++i) {
    const int row = i * RPI + r;
    kr[i] = row < len ? *reinterpret_cast<const uint4*>(kbase + (int64_t)row * D)
                      : make_uint4(0u, 0u, 0u, 0u);
  }
#pragma unroll
  for (int i = 0; i < ITER; ++i) {
    const int row = i * RPI + r;
    vr[i] = row < len ? *reinterpret_cast<const uint4*>(vbase + (int64_t)row * D)
                      : make_uint4(0u, 0u, 0u, 0u);
  }

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
  float m[G], p[G], l[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = wave_max(mine_ok ? lg[g] : -INFINITY);
    p[g] = mine_ok ? fast_exp2(lg[g] - m[g]) : 0.f;
    l[g] = wave_sum(p[g]);
  }

  float acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
#pragma unroll
  for (int i = 0; i < ITER; ++i) {
    float vf[EPL];
    unpack16<T>(vr[i], vf);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float pb = __shfl(p[g], r * LPR + i);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(pb, vf[e], acc[g][e]);
    }
  }
#pragma unroll
  for (int msk = LPR; msk < kWave; msk <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] += __shfl_xor(acc[g][e], msk);

  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) wacc[wave][g][jj * EPL + e] = acc[g][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = m[g]; wl[wave][g] = l[g]; }
  }
  __syncthreads();

  float* dst = part + ((bh * maxwg + j) * G) * (int64_t)PSTRIDE;
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
    dst[g * PSTRIDE + 4 + e] = a;
    if (e == 0) { dst[g * PSTRIDE] = M; dst[g * PSTRIDE + 1] = L; }
  }
}

// ---------------------------------------------------------------------------
// k_combine: merge the partials of each (b, q head)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(64) void k_combine(const float* __restrict__ part,
                                                const int* __restrict__ ucnt,
                                                T* __restrict__ out, int Hq,
                                                int Hkv, int G,
                                                int tiles_per_seg,
                                                int win_tiles, int maxwg) {
  constexpr int PSTRIDE = D + 4;
  constexpr int DPT = D / 64;
  const int64_t bhq = blockIdx.x;
  const int64_t b = bhq / Hq, hq = bhq % Hq;
  const int64_t hk = hq / G;
  const int g = (int)(hq % G);
  const int64_t bh = b * Hkv + hk;
  const int total = ucnt[bh] * tiles_per_seg + win_tiles;
  const int nwg = (total + 3) / 4;
  const float* src = part + ((bh * maxwg) * G + g) * (int64_t)PSTRIDE;
  const int64_t wstride = (int64_t)G * PSTRIDE;
  float M = -INFINITY;
  for (int w = 0; w < nwg; ++w) M = fmaxf(M, src[w * wstride]);
  float L = 0.f, a[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) a[i] = 0.f;
  for (int w = 0; w < nwg; ++w) {
    const float* pw = src + w * wstride;
    const float f = fast_exp2(pw[0] - M);
    L = fmaf(pw[1], f, L);
#pragma unroll
    for (int i = 0; i < DPT; ++i) a[i] = fmaf(pw[4 + threadIdx.x + 64 * i], f, a[i]);
  }
  const float inv = 1.f / L;
#pragma unroll
  for (int i = 0; i < DPT; ++i)
    out[bhq * D + threadIdx.x + 64 * i] = from_f32<T>(a[i] * inv);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
thread_local char g_last_error[256] = "";


// ---- launch helper with optional per-kernel event timing -----------------
// While profiling is enabled on a host thread, every launch goes through
// hipExtLaunchKernelGGL with a start/stop event pair, so the recorded times
// bracket exactly that kernel's execution on its stream.
struct Profiler {
  bool on = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
};
thread_local Profiler g_prof;

template <typename F, typename... Args>
void launch(int kind, F kern, dim3 grid, dim3 block, size_t shm, hipStream_t st,
            Args... args) {
  if (g_prof.on) {
    hipEvent_t a = nullptr, b = nullptr;
    if (hipEventCreate(&a) == hipSuccess && hipEventCreate(&b) == hipSuccess) {
      hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)shm, st, a, b, 0u, args...);
      g_prof.recs.push_back({kind, a, b});
      return;
    }
  }
  hipLaunchKernelGGL(kern, grid, block, shm, st, args...);
}

struct Shape {
  int B, Hq, Hkv, G, d, n, c, w;
  int64_t cap, s_cap;
  radar_dtype dt;
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

radar_status check_cfg(const radar_config* cfg, Shape* s) {
  if (!cfg) return RADAR_EINVAL;
  if (cfg->batch < 1 || cfg->n_q_heads < 1 || cfg->n_kv_heads < 1 ||
      cfg->seg_len < 1 || cfg->window < 0 || cfg->capacity < 1 ||
      cfg->n_q_heads % cfg->n_kv_heads != 0)
    return RADAR_EINVAL;
  if (cfg->kv_dtype != RADAR_F32 && cfg->kv_dtype != RADAR_BF16) return RADAR_EINVAL;
  const int G = cfg->n_q_heads / cfg->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return RADAR_EUNSUPPORTED;
  if (cfg->head_dim != 64 && cfg->head_dim != 128) return RADAR_EUNSUPPORTED;
  const int n = cfg->n_features;
  if (n != 64 && n != 128 && n != 256 && n != 512) return RADAR_EUNSUPPORTED;
  if (cfg->capacity > (int64_t)1 << 31) return RADAR_EUNSUPPORTED;
  s->B = cfg->batch; s->Hq = cfg->n_q_heads; s->Hkv = cfg->n_kv_heads; s->G = G;
  s->d = cfg->head_dim; s->n = n; s->c = cfg->seg_len; s->w = cfg->window;
  s->cap = cfg->capacity; s->s_cap = cfg->capacity / cfg->seg_len;
  s->dt = cfg->kv_dtype;
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
  const int64_t wt = ceil_div(wmax, kTile);
  L.maxwg = (int)ceil_div((int64_t)L.umax * L.tiles_per_seg + wt, 4);
  size_t off = 0;
  L.phiq = off;   off += align256((size_t)s.B * s.Hq * s.n * 4);
  L.scores = off; off += align256((size_t)s.B * s.Hq * std::max<int64_t>(1, s.s_cap) * 4);
  L.uni = off;    off += align256((size_t)s.B * s.Hkv * L.umax * 4);
  L.ucnt = off;   off += align256((size_t)s.B * s.Hkv * 4);
  L.part = off;   off += align256((size_t)s.B * s.Hkv * L.maxwg * s.G * (s.d + 4) * 4);
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
radar_status launch_build_t(const Shape& s, const void* K, const float* omega,
                            float* summ, int seg_first, int seg_count,
                            hipStream_t st) {
  const int slices = s.n / (64 * FT);
  const int64_t items = (int64_t)s.B * s.Hkv * seg_count;
  if (items == 0) return RADAR_OK;
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
                     reinterpret_cast<const T*>(K), omega, summ, s.n, s.c, s.cap,
                     s.s_cap, seg_first, seg_count, items, s1, s2, out_scale, s.cap);
  return launch_status();
}

template <typename T, int D>
radar_status launch_build_d(const Shape& s, const void* K, const float* omega,
                            float* summ, int seg_first, int seg_count,
                            hipStream_t st) {
  // features per workgroup = 64 * FT; FT capped so the resident Omega slice
  // stays at 128 VGPRs or fewer
  constexpr int FTMAX = (D * sizeof(T) <= 256) ? 8 : 4;
  const int ft = std::min(s.n / 64, FTMAX);
  switch (ft) {
    case 1: return launch_build_t<T, D, 1>(s, K, omega, summ, seg_first, seg_count, st);
    case 2: return launch_build_t<T, D, 2>(s, K, omega, summ, seg_first, seg_count, st);
    case 4: return launch_build_t<T, D, 4>(s, K, omega, summ, seg_first, seg_count, st);
    default:
      if constexpr (FTMAX >= 8)
        return launch_build_t<T, D, 8>(s, K, omega, summ, seg_first, seg_count, st);
      return RADAR_EUNSUPPORTED;
  }
}

radar_status launch_build(const Shape& s, const void* K, const float* omega,
                          float* summ, int seg_first, int seg_count,
                          hipStream_t st) {
  if (s.dt == RADAR_BF16)
    return s.d == 64 ? launch_build_d<bf16_t, 64>(s, K, omega, summ, seg_first, seg_count, st)
                     : launch_build_d<bf16_t, 128>(s, K, omega, summ, seg_first, seg_count, st);
  return s.d == 64 ? launch_build_d<float, 64>(s, K, omega, summ, seg_first, seg_count, st)
                   : launch_build_d<float, 128>(s, K, omega, summ, seg_first, seg_count, st);
}

// ---- decode pieces -------------------------------------------------------
template <typename T, int D>
void launch_phi_q(const Shape& s, const void* q, const float* omega, float* phiq,
                  hipStream_t st) {
  const float s1 = kLog2e / std::pow((float)s.d, 0.25f);
  const float s2 = kLog2e / (2.f * std::sqrt((float)s.d));
  launch(RADAR_K_PHI_Q, k_phi_q<T, D>, dim3((unsigned)(s.B * s.Hq)), dim3(256), 0, st,
                     reinterpret_cast<const T*>(q), omega, phiq, s.n, s1, s2,
                     1.f / std::sqrt((float)s.n));
}

template <int N>
void launch_score_n(const Shape& s, const float* phiq, const float* summ,
                    float* scores, int n_cand, hipStream_t st) {
  const dim3 grid((unsigned)ceil_div(n_cand, 64), (unsigned)(s.B * s.Hkv));
  const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);
  switch (s.G) {
    case 1: launch(RADAR_K_SCORE, k_score<N, 1>, grid, dim3(256), 0, st, phiq, summ, scores, s.Hq, s.Hkv, n_cand, s.s_cap, nc_cap); break;
    case 2: launch(RADAR_K_SCORE, k_score<N, 2>, grid, dim3(256), 0, st, phiq, summ, scores, s.Hq, s.Hkv, n_cand, s.s_cap, nc_cap); break;
    case 4: launch(RADAR_K_SCORE, k_score<N, 4>, grid, dim3(256), 0, st, phiq, summ, scores, s.Hq, s.Hkv, n_cand, s.s_cap, nc_cap); break;
    default: launch(RADAR_K_SCORE, k_score<N, 8>, grid, dim3(256), 0, st, phiq, summ, scores, s.Hq, s.Hkv, n_cand, s.s_cap, nc_cap); break;
  }
}

void launch_score(const Shape& s, const float* phiq, const float* summ,
                  float* scores, int n_cand, hipStream_t st) {
  switch (s.n) {
    case 64: launch_score_n<64>(s, phiq, summ, scores, n_cand, st); break;
    case 128: launch_score_n<128>(s, phiq, summ, scores, n_cand, st); break;
    case 256: launch_score_n<256>(s, phiq, summ, scores, n_cand, st); break;
    default: launch_score_n<512>(s, phiq, summ, scores, n_cand, st); break;
  }
}

template <typename T, int D, int G>
void launch_attend_g(const Shape& s, const void* q, const void* K, const void* V,
                     const int* uni, const int* ucnt, float* part,
                     const WsLayout& L, int grid_x, int64_t ws, int64_t t,
                     hipStream_t st) {
  const float qscale = kLog2e / std::sqrt((float)s.d);
  launch(RADAR_K_ATTEND, k_attend<T, D, G>, dim3((unsigned)grid_x, (unsigned)(s.B * s.Hkv)),
                     dim3(256), 0, st, reinterpret_cast<const T*>(q),
                     reinterpret_cast<const T*>(K), reinterpret_cast<const T*>(V),
                     uni, ucnt, part, s.Hq, s.Hkv, s.cap, s.c, L.tiles_per_seg, ws,
                     t, L.umax, L.maxwg, qscale);
}

template <typename T, int D>
void launch_attend_d(const Shape& s, const void* q, const void* K, const void* V,
                     const int* uni, const int* ucnt, float* part,
                     const WsLayout& L, int grid_x, int64_t ws, int64_t t,
                     hipStream_t st) {
  switch (s.G) {
    case 1: launch_attend_g<T, D, 1>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st); break;
    case 2: launch_attend_g<T, D, 2>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st); break;
    case 4: launch_attend_g<T, D, 4>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st); break;
    default: launch_attend_g<T, D, 8>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st); break;
  }
}

template <typename T, int D>
void launch_combine_d(const Shape& s, const float* part, const int* ucnt, void* out,
                      const WsLayout& L, int win_tiles, hipStream_t st) {
  launch(RADAR_K_COMBINE, k_combine<T, D>, dim3((unsigned)(s.B * s.Hq)), dim3(64), 0, st,
                     part, ucnt, reinterpret_cast<T*>(out), s.Hq, s.Hkv, s.G,
                     L.tiles_per_seg, win_tiles, L.maxwg);
}

// exact attention over the union written to the workspace, then combine
radar_status attend_and_combine(const Shape& s, const void* q, const void* K,
                                const void* V, int u_bound, int64_t ws, int64_t t,
                                void* out, unsigned char* w, const WsLayout& L,
                                hipStream_t st) {
  const int* uni = reinterpret_cast<const int*>(w + L.uni);
  const int* ucnt = reinterpret_cast<const int*>(w + L.ucnt);
  float* part = reinterpret_cast<float*>(w + L.part);
  const int win_tiles = (int)ceil_div(t - ws, kTile);
  const int grid_x = (int)ceil_div((int64_t)u_bound * L.tiles_per_seg + win_tiles, 4);
  if (s.dt == RADAR_BF16) {
    if (s.d == 64) {
      launch_attend_d<bf16_t, 64>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st);
      launch_combine_d<bf16_t, 64>(s, part, ucnt, out, L, win_tiles, st);
    } else {
      launch_attend_d<bf16_t, 128>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st);
      launch_combine_d<bf16_t, 128>(s, part, ucnt, out, L, win_tiles, st);
    }
  } else {
    if (s.d == 64) {
      launch_attend_d<float, 64>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st);
      launch_combine_d<float, 64>(s, part, ucnt, out, L, win_tiles, st);
    } else {
      launch_attend_d<float, 128>(s, q, K, V, uni, ucnt, part, L, grid_x, ws, t, st);
      launch_combine_d<float, 128>(s, part, ucnt, out, L, win_tiles, st);
    }
  }
  return launch_status();
}

void window_split(const Shape& s, int64_t t, int64_t* ws, int* n_cand) {
  const int64_t past = std::max<int64_t>(0, t - s.w);
  *ws = (int64_t)s.c * (past / s.c);
  *n_cand = (int)(*ws / s.c);
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

int32_t radar_abi_version(void) { return RADAR_ABI_VERSION; }

radar_status radar_profile_enable(int32_t on) {
  g_prof.on = on != 0;
  return RADAR_OK;
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
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
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
    case RADAR_EUNSUPPORTED: return "shape not supported by this build";
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
                               const float* omega, int64_t t, float* summaries,
                               hipStream_t stream) {
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (!K || !omega || !summaries) return RADAR_EINVAL;
  if (!aligned16(K) || !aligned16(omega) || !aligned16(summaries)) return RADAR_EINVAL;
  if (t < 1 || t > s.cap) return RADAR_ECAPACITY;
  const int64_t n_seg = t / s.c;
  if (n_seg == 0) return RADAR_OK;
  return launch_build(s, K, omega, summaries, 0, (int)n_seg, stream);
}

radar_status radar_append(const radar_config* cfg, void* K, void* V,
                          const void* k_new, const void* v_new,
                          const float* omega, int64_t t, float* summaries,
                          hipStream_t stream) {
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (!K || !V || !k_new || !v_new || !omega || !summaries) return RADAR_EINVAL;
  if (!aligned16(K) || !aligned16(V) || !aligned16(k_new) || !aligned16(v_new) ||
      !aligned16(omega) || !aligned16(summaries))
    return RADAR_EINVAL;
  if (t < 0 || t >= s.cap) return RADAR_ECAPACITY;
  const unsigned grid = (unsigned)(s.B * s.Hkv);
  if (s.dt == RADAR_BF16) {
    if (s.d == 64)
      launch(RADAR_K_APPEND, k_append<bf16_t, 64>, dim3(grid), dim3(64), 0, stream,
                         (bf16_t*)K, (bf16_t*)V, (const bf16_t*)k_new, (const bf16_t*)v_new, s.cap, t);
    else
      launch(RADAR_K_APPEND, k_append<bf16_t, 128>, dim3(grid), dim3(64), 0, stream,
                         (bf16_t*)K, (bf16_t*)V, (const bf16_t*)k_new, (const bf16_t*)v_new, s.cap, t);
  } else {
    if (s.d == 64)
      launch(RADAR_K_APPEND, k_append<float, 64>, dim3(grid), dim3(64), 0, stream,
                         (float*)K, (float*)V, (const float*)k_new, (const float*)v_new, s.cap, t);
    else
      launch(RADAR_K_APPEND, k_append<float, 128>, dim3(grid), dim3(64), 0, stream,
                         (float*)K, (float*)V, (const float*)k_new, (const float*)v_new, s.cap, t);
  }
  r = launch_status();
  if (r != RADAR_OK) return r;
  if ((t + 1) % s.c == 0) {
    const int seg = (int)((t + 1) / s.c - 1);
    return launch_build(s, K, omega, summaries, seg, 1, stream);
  }
  return RADAR_OK;
}

radar_status radar_decode(const radar_config* cfg, const void* q, const void* K,
                          const void* V, const float* omega,
                          const float* summaries, int64_t t, int32_t k,
                          void* out, int32_t* selected, float* scores,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (!q || !K || !V || !omega || !summaries || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(omega) ||
      !aligned16(summaries) || !aligned16(out) ||
      (selected && !aligned16(selected)) || (scores && !aligned16(scores)))
    return RADAR_EINVAL;
  if (k < 1 || k > kMaxK) return RADAR_EUNSUPPORTED;
  if (t < 1 || t > s.cap) return RADAR_ECAPACITY;
  const WsLayout L = ws_layout(s, k);
  if (!workspace || !aligned16(workspace)) return RADAR_EWORKSPACE;
  if (workspace_bytes < L.total) return RADAR_EWORKSPACE;
  int64_t ws;
  int n_cand;
  window_split(s, t, &ws, &n_cand);
  if (n_cand > kMaxCand) return RADAR_EUNSUPPORTED;
  const int k_eff = std::min(k, n_cand);

  unsigned char* w = reinterpret_cast<unsigned char*>(workspace);
  float* phiq = reinterpret_cast<float*>(w + L.phiq);
  float* sc = reinterpret_cast<float*>(w + L.scores);
  int* uni = reinterpret_cast<int*>(w + L.uni);
  int* ucnt = reinterpret_cast<int*>(w + L.ucnt);
  const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);

  if (n_cand > 0) {
    if (s.dt == RADAR_BF16) {
      if (s.d == 64) launch_phi_q<bf16_t, 64>(s, q, omega, phiq, stream);
      else launch_phi_q<bf16_t, 128>(s, q, omega, phiq, stream);
    } else {
      if (s.d == 64) launch_phi_q<float, 64>(s, q, omega, phiq, stream);
      else launch_phi_q<float, 128>(s, q, omega, phiq, stream);
    }
    launch_score(s, phiq, summaries, sc, n_cand, stream);
  }
  const int npl = std::max(1, (n_cand + 63) / 64);
  launch(RADAR_K_TOPK, k_topk_union, dim3((unsigned)(s.B * s.Hkv)), dim3(256),
                     (size_t)4 * npl * 64 * sizeof(float), stream, sc, s.Hq, s.Hkv,
                     s.G, n_cand, nc_cap, k, k_eff, uni, ucnt, L.umax, selected,
                     scores, nullptr, 0);
  r = launch_status();
  if (r != RADAR_OK) return r;
  const int u_bound = std::min(s.G * k_eff, n_cand);
  return attend_and_combine(s, q, K, V, u_bound, ws, t, out, w, L, stream);
}

radar_status radar_attend_selected(const radar_config* cfg, const void* q,
                                   const void* K, const void* V,
                                   const int32_t* selected, int32_t k, int64_t t,
                                   void* out, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (!q || !K || !V || !selected || !out) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(selected) ||
      !aligned16(out))
    return RADAR_EINVAL;
  if (k < 1 || k > kMaxK) return RADAR_EUNSUPPORTED;
  if (t < 1 || t > s.cap) return RADAR_ECAPACITY;
  const WsLayout L = ws_layout(s, k);
  if (!workspace || !aligned16(workspace)) return RADAR_EWORKSPACE;
  if (workspace_bytes < L.total) return RADAR_EWORKSPACE;
  int64_t ws;
  int n_cand;
  window_split(s, t, &ws, &n_cand);
  unsigned char* w = reinterpret_cast<unsigned char*>(workspace);
  int* uni = reinterpret_cast<int*>(w + L.uni);
  int* ucnt = reinterpret_cast<int*>(w + L.ucnt);
  launch(RADAR_K_TOPK, k_topk_union, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0, stream,
                     nullptr, s.Hq, s.Hkv, s.G, n_cand, 1, k, 0, uni, ucnt, L.umax,
                     nullptr, nullptr, selected, k);
  r = launch_status();
  if (r != RADAR_OK) return r;
  const int u_bound = std::min(s.G * k, n_cand);
  return attend_and_combine(s, q, K, V, u_bound, ws, t, out, w, L, stream);
}

}  // extern "C"

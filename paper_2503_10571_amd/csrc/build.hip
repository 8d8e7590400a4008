// Index build (Eq. 4 and Eq. 5): k_build and its launcher. The segment
// close of an append runs the same kernel on one segment, so appends and
// rebuilds agree bit for bit.
#include "radar_impl.h"

namespace radar_impl {

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

template <typename T, int D, int TL>
struct BuildTile {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kPitch = kRowBytes + 16;          // LDS row pitch
  static constexpr int kChunksPerRow = kRowBytes / 16;
  static constexpr int kChunksPerThread = TL * kChunksPerRow / 256;
};

// TL: keys per LDS tile (64, or 128 for bf16 keys in segments of >= 128)
template <typename T, int D, int FT, int TL>
__global__ __launch_bounds__(256) void k_build(
    const T* __restrict__ K, const void* __restrict__ omega, bool obf,
    float* __restrict__ summ, int n, int c, int64_t cap, int64_t s_cap,
    int seg_first, int seg_count, int64_t n_items, float s1, float s2,
    float out_scale, int64_t kv_head_stride_rows,
    const int64_t* __restrict__ pos, int Hkv, int n_sink) {
  using MC = MfmaCfg<T>;
  using BT = BuildTile<T, D, TL>;
  constexpr int KB = D / MC::kK;
  constexpr int CPR = BT::kChunksPerRow;
  constexpr int CPT = BT::kChunksPerThread;
  static_assert(CPT >= 1 && (256 % CPR) == 0, "tile shape");

  __shared__ __attribute__((aligned(16))) unsigned char tile_lds[2][TL * BT::kPitch];
  __shared__ float nrm_lds[2][TL];

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

  const int ntiles = (c + TL - 1) / TL;
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
    pre_valid = min(TL, c - tl_ * TL);
    const T* src = base + (int64_t)tl_ * TL * D;
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
        if constexpr (CPR == 32) sq = xor_sum<16>(sq);
      }
      if (ch == 0) nrm_lds[buf][row] = sq * s2;
    }
  };

  // 16-token sub-tiles of the tile in `buf`; FULL: no rows to mask
  auto compute = [&](int buf, int valid, auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    const unsigned char* tb = tile_lds[buf];
#pragma unroll
    for (int st = 0; st < TL / 16; ++st) {
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

    if (valid == TL) compute(buf, valid, std::true_type{});
    else compute(buf, valid, std::false_type{});

    if (tl == ntiles - 1) {                // segment complete
      const int64_t bh = (uint32_t)item / (uint32_t)seg_count;
      const int64_t sg = seg_of(item);
      float* dst = summ + (bh * s_cap + sg) * n + fbase;
#pragma unroll
      for (int f = 0; f < FT; ++f) {
        float v = psum[f];
        v = xor_sum<16>(v);
        v = xor_sum<32>(v);
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

template <typename T, int D, int FT, int TL>
radar_status launch_build_tl(const Shape& s, const void* K, const void* omega,
                             float* summ, int seg_first, int seg_count,
                             const int64_t* pos, hipStream_t st) {
  const int slices = s.n / (64 * FT);
  const int64_t items = (int64_t)s.B * s.Hkv * seg_count;
  if (items == 0) return RADAR_OK;
  if (items >= ((int64_t)1 << 31)) return RADAR_EUNSUPPORTED;   // 32-bit item ids
  auto kern = k_build<T, D, FT, TL>;
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

// 128-key tiles halve the tile loop's barriers and prefetch rounds per key
// (same sums in the same order: each lane's column sums run over the same
// 16-key sub-tiles); for bf16 keys only (fp32 rows at d = 128 would need
// 136 KB of LDS) and segments of at least 128 keys (shorter ones would run
// half-empty tiles)
template <typename T, int D, int FT>
radar_status launch_build_t(const Shape& s, const void* K, const void* omega,
                            float* summ, int seg_first, int seg_count,
                            const int64_t* pos, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (s.c >= 128)
      return launch_build_tl<T, D, FT, 128>(s, K, omega, summ, seg_first, seg_count, pos, st);
  }
  return launch_build_tl<T, D, FT, 64>(s, K, omega, summ, seg_first, seg_count, pos, st);
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
}  // namespace radar_impl

// The fused decode kernel (phi(q), scores, top-k, union, attention and merge
// of one (b, kv head) in R workgroups) and its select-only instantiation,
// for one feature count: this unit is compiled once per n with
// -DRADAR_FUSED_N=<n>, so the instantiations build in parallel.
#include "radar_impl.h"

#ifndef RADAR_FUSED_N
#error "compile with -DRADAR_FUSED_N=<feature count>"
#endif

namespace radar_impl {

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
// MODE kFusedSelect stops after phase 4 and writes the union to uni_out /
// ucnt_out for the split path's attention (the select path: one workgroup
// per pair replaces the phi(q), score and top-k kernels). MODE kFusedScored
// starts at phase 3: the scores of phases 1-2 come from the split path's
// chip-wide phi(q) and score kernels (gscores [B][Hq][nc_cap]), for pairs
// whose summary rows are too many to read R times (the scored path).

template <typename T, int D, int G, int N, int MODE>
__global__ __launch_bounds__(512) void k_decode_fused(
    const T* __restrict__ q, const T* __restrict__ K, const T* __restrict__ V,
    const void* __restrict__ omega, bool obf, const float* __restrict__ summ,
    T* __restrict__ out, int32_t* __restrict__ selected,
    float* __restrict__ sel_scores, int Hq, int Hkv, int64_t cap,
    int64_t s_cap, int tiles_per_seg, SeqArgs sa, int per_head, float s1,
    float s2, float inv_sqrt_n, float qscale, int* __restrict__ uni_out,
    int* __restrict__ ucnt_out, int umax, AppendArgs ap, int R, int n_pairs,
    float* __restrict__ part, int maxwg, const float* __restrict__ gscores,
    int nc_cap, uint64_t* __restrict__ clk, int clk_max) {
  constexpr bool SEL = MODE == kFusedSelect;
  constexpr bool SCORED = MODE == kFusedScored;
  constexpr int NW = kFusedWaves;
  constexpr int QPL = D / 16;              // q elements per lane (phase 1)
  constexpr int FPL = N / 64;              // features per lane (phase 2)
  using TA = TileAttn<T, D, G>;
  constexpr int EPL = TA::EPL, LPR = TA::LPR;
  constexpr int SEL_FLOATS = SCORED ? 0 : G * N + G * kFusedMaxCand;
  constexpr int MRG_FLOATS = NW * G * D;
  constexpr int AREA = SEL_FLOATS > MRG_FLOATS ? SEL_FLOATS : MRG_FLOATS;
  static_assert(G <= kFusedMaxG, "group");
  static_assert(N % (4 * NW) == 0, "features");

  // phi(q) and the scores live only until the top-k; the merge reuses them
  __shared__ __attribute__((aligned(16))) float area[AREA];
  __shared__ int sel_lds[G * kMaxK];
  __shared__ unsigned bits_lds[G * kBitmapWords];
  __shared__ int uni_lds[G * kMaxK];
  __shared__ u64 list_lds[G][kMaxK];
  __shared__ float wm[NW][G], wl[NW][G];
  __shared__ int ucnt_lds;
  float* phq = area;                       // [G][N]
  float* sc = area + G * N;                // [G][kFusedMaxCand]
  float* wacc = area;                      // [NW][G][D]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // measurement hook: the first thread stamps the phase boundaries (every
  // stamp starts as the entry time: phases 1-2 when they do not run keep it;
  // later stamps are written on every path)
  const bool clocked = clk != nullptr && (int)blockIdx.x < clk_max;   // uniform
  uint64_t* const cw = clk + (clocked ? (int64_t)blockIdx.x * RADAR_CLOCK_STAMPS : 0);
  auto stamp = [&](int i) {
    if (clocked && tid == 0) cw[i] = (uint64_t)wall_clock64();
  };
  if (clocked && tid == 0) {
    const uint64_t t0 = (uint64_t)wall_clock64();
#pragma unroll
    for (int i = 0; i < RADAR_CLOCK_STAMPS; ++i) cw[i] = t0;
  }
  // workgroup rj < R of pair bh: the workgroups of a pair differ by a
  // multiple of n_pairs, so they share an XCD (and its L2) when n_pairs is a
  // multiple of 8 (dealing a pair's workgroups over all XCDs instead measured
  // 2% slower on the scored path at 512K)
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
  // phases 1 and 2, or this one when there are no candidates (or no phases
  // 1 and 2).
  if (ap.K) {                              // uniform
    if (wave == NW - 1) append_row(ap, cap, bh, Hkv, lane);
    if (n_cand == 0 || SCORED) __syncthreads();
  }

  if constexpr (!SCORED) {
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
    stamp(1);

    // ---- 2. scores ------------------------------------------------------
    if constexpr (N > 512) {
      // each 16-row batch in chunks of FC features per lane (chunk ch of
      // lane l: features ch * 64 * FC + l * FC + e), the chunk layout of
      // the split path's score kernel, so a lane holds one chunk of the
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
          v = xor_sum<16>(v);
          v = xor_sum<32>(v);
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
            v = xor_sum<16>(v);
            v = xor_sum<32>(v);
            if (lane < 16 && row < n_cand) sc[g * kFusedMaxCand + row] = v;
          }
        }
      }
    }
    __syncthreads();
    stamp(2);
  }
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
    const float* src = SCORED ? gscores + (b * Hq + hq) * (int64_t)nc_cap
                              : sc + wave * kFusedMaxCand;
    int* row = sel_lds + wave * k_eff;
    u64* list = list_lds[wave];
    const int npl = (n_cand + 63) / 64;
    if (npl <= 1) head_topk<1>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 2) head_topk<2>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 4) head_topk<4>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 8) head_topk<8>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (!SCORED || npl <= 16)
      head_topk<16>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if constexpr (SCORED)             // up to 2048 candidates
      head_topk<32>(src, n_cand, k, k_eff, row, so, sco, lane, list);
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
  stamp(3);

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
  stamp(4);
  if constexpr (SEL) {                     // hand the union to the split path
    for (int i = tid; i < n_segs; i += NW * 64) uni_out[bh * umax + i] = segs[i];
    if (tid == 0) ucnt_out[bh] = n_segs;
    stamp(5);
    stamp(6);
    return;
  }
  const int seg_tiles = n_segs * tiles_per_seg;

  // ---- 5. segment tiles ---------------------------------------------------
  // (64-row tiles dealt round robin over the pair's waves; equal shares of
  // rows instead, cut at segment ends, measured slower: the shares start
  // mid-tile, so waves run more partial tiles, each costing nearly a whole
  // one)
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
  stamp(5);
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
  if (clocked) {
    __syncthreads();
    stamp(6);
  }
}

// The launch helpers below are compiled once per unit, each with its own
// RADAR_FUSED_N: internal linkage keeps the units' copies apart.
namespace {

template <typename T, int D, int G, int MODE>
radar_status launch_fused_tdg(const FusedArgs& a) {
  const Shape& s = *a.s;
  // the scored kernel reads no summaries: one instantiation serves every n
  constexpr int N = MODE == kFusedScored ? 64 : RADAR_FUSED_N;
  const float s1 = kLog2e / std::pow((float)s.d, 0.25f);
  const float s2 = kLog2e / (2.f * std::sqrt((float)s.d));
  const int n_pairs = s.B * s.Hkv;
  const int kind = MODE == kFusedSelect ? RADAR_K_SELECT
                   : MODE == kFusedScored ? RADAR_K_SCORED : RADAR_K_FUSED;
  launch(kind, k_decode_fused<T, D, G, N, MODE>,
         dim3((unsigned)(n_pairs * a.R)), dim3(kFusedWaves * 64), 0, a.st,
         reinterpret_cast<const T*>(a.q), reinterpret_cast<const T*>(a.K),
         reinterpret_cast<const T*>(a.V), a.omega, s.obf, a.summ,
         reinterpret_cast<T*>(a.out), a.selected, a.sel_scores, s.Hq, s.Hkv, s.cap,
         s.s_cap, (int)ceil_div(s.c, kTile), a.sa, s.per_head, s1, s2,
         1.f / std::sqrt((float)s.n), kLog2e / std::sqrt((float)s.d), a.uni_out,
         a.ucnt_out, a.umax, a.ap, a.R, n_pairs, a.part, a.maxwg, a.gscores, a.nc_cap,
         g_clock, g_clock_max);
  return launch_status();
}

template <typename T, int D, int MODE>
radar_status launch_fused_td(const FusedArgs& a) {
  switch (a.s->G) {
    case 1: return launch_fused_tdg<T, D, 1, MODE>(a);
    case 2: return launch_fused_tdg<T, D, 2, MODE>(a);
    default: return launch_fused_tdg<T, D, 4, MODE>(a);
  }
}

// fp32 caches with d = 128 have no fused or scored instantiation (their
// tiles need more registers than the fused kernel has to spare): the select
// kernel serves them, and the host never asks for the others
template <int MODE>
radar_status launch_fused_mode(const FusedArgs& a) {
  const Shape& s = *a.s;
  if (s.dt == RADAR_BF16)
    return s.d == 64 ? launch_fused_td<bf16_t, 64, MODE>(a) : launch_fused_td<bf16_t, 128, MODE>(a);
  if (s.d == 64) return launch_fused_td<float, 64, MODE>(a);
  if constexpr (MODE == kFusedSelect) return launch_fused_td<float, 128, kFusedSelect>(a);
  return RADAR_EUNSUPPORTED;
}

}  // namespace

#define RADAR_FUSED_ENTRY2(n) launch_fused_n##n
#define RADAR_FUSED_ENTRY(n) RADAR_FUSED_ENTRY2(n)
radar_status RADAR_FUSED_ENTRY(RADAR_FUSED_N)(const FusedArgs& a, bool sel) {
  return sel ? launch_fused_mode<kFusedSelect>(a) : launch_fused_mode<kFusedFull>(a);
}

#if RADAR_FUSED_N == 64
radar_status launch_fused_scored(const FusedArgs& a) {
  return launch_fused_mode<kFusedScored>(a);
}
#endif

}  // namespace radar_impl

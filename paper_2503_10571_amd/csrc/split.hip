// The split decode path's stages, each spread over the whole chip: phi(q),
// Eq. 6 scores, the exact segment mass, top-k and union, the given-selection
// union, the gather attention and the merge of its partials (also used by
// the fused path when several workgroups share a pair).
#include "radar_impl.h"

namespace radar_impl {

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
// k_score: a[h][s] = phi(q_h) . summ[s], Eq. 6
// ---------------------------------------------------------------------------
// Workgroup = 1, 2 or 4 waves x (16 * RB) summary rows of one (b, kv head)
// (fewer waves per workgroup when that spreads a small call over more CUs;
// the waves are independent). Lane l holds FPL = n / 64 features of phi(q)
// for the G heads of the group, in chunks of at most 8 (n = 1024 and 2048
// take 2 to 8 chunks, so the rows of a batch fit in registers); each chunk
// of a row is one contiguous wave load, and all of a batch's rows are loaded
// before any is reduced. A 16-row batch is transpose-reduced inside each
// 16-lane row with DPP, then summed over the four rows.
// With S > 1 the S waves of a workgroup share one batch of rows instead and
// each takes NCH / S of the chunks (one round trip to memory instead of
// NCH / 2 for a wave that walks them all); the waves' row sums are added in
// LDS in wave order.
template <int N, int G, int S>
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
  static_assert(NCH % S == 0 && (S == 1 || RB == 1), "feature split");
  constexpr int CPW = NCH / S;             // chunks of each wave
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bh = blockIdx.y;
  const int64_t b = bh / Hkv, hk = bh % Hkv;
  const int n_cand = seq_span(sa, b).n_cand;
  const int wrow0 = S > 1 ? blockIdx.x * 16
                          : (blockIdx.x * (blockDim.x >> 6) + wave) * (16 * RB);
  // wave-uniform, and workgroup-uniform with S > 1 (the waves share rows),
  // so the barrier below is reached by all waves or by none
  if (wrow0 >= n_cand) return;
  const int ch0 = S > 1 ? wave * CPW : 0;  // this wave's first chunk

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
  // a chunk's phi(q) features and rows
  auto load_chunk = [&](int ch, float (&pq)[G][FC], float (&x)[RB][16][FC]) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* src = phiq + ((b * Hq + hk * G + g) * N) + ch * 64 * FC + lane * FC;
#pragma unroll
      for (int e = 0; e < FC; ++e) pq[g][e] = src[e];
    }
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
  };
  auto add_chunk = [&](const float (&pq)[G][FC], const float (&x)[RB][16][FC]) {
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
  };
  // Several chunks at G = 4 (four features per lane): two chunks in flight,
  // the next one's loads issued before this one's products (same products,
  // same order; 376 registers, one wave per SIMD, as these launches run);
  // otherwise one chunk's rows live at a time (G = 8 would not fit).
  constexpr bool kTwo = CPW > 1 && CPW % 2 == 0 && FC == 4 && G == 4;
  if constexpr (kTwo) {
    float pqa[G][FC], xa[RB][16][FC], pqb[G][FC], xb[RB][16][FC];
    load_chunk(ch0, pqa, xa);
#pragma unroll 1
    for (int ch = ch0; ch < ch0 + CPW; ch += 2) {
      load_chunk(ch + 1, pqb, xb);
      __builtin_amdgcn_sched_barrier(0);
      add_chunk(pqa, xa);
      if (ch + 2 < ch0 + CPW) load_chunk(ch + 2, pqa, xa);
      __builtin_amdgcn_sched_barrier(0);
      add_chunk(pqb, xb);
    }
  } else {
#pragma unroll 1
    for (int ch = ch0; ch < ch0 + CPW; ++ch) {
      float pq[G][FC], x[RB][16][FC];
      load_chunk(ch, pq, x);
      // with several chunks the compiler would sink each load to its first
      // use and wait on one load at a time; keep the chunk's loads together
      if constexpr (CPW > 1) __builtin_amdgcn_sched_barrier(0);
      add_chunk(pq, x);
    }
  }
  __shared__ float red[S > 1 ? S : 1][G][16];
#pragma unroll
  for (int bt = 0; bt < RB; ++bt) {
    const int row = wrow0 + bt * 16 + (lane & 15);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      transpose_reduce<16>(part[bt][g], lane);
      float v = part[bt][g][0];
      v = xor_sum<16>(v);
      v = xor_sum<32>(v);
      if constexpr (S > 1) {
        if (lane < 16) red[wave][g][lane] = v;
      } else {
        if (lane < 16 && row < n_cand)
          scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + row] = v;
      }
    }
  }
  if constexpr (S > 1) {
    __syncthreads();
    if (wave == 0 && lane < 16 && wrow0 + lane < n_cand) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float v = red[0][g][lane];
#pragma unroll
        for (int w = 1; w < S; ++w) v += red[w][g][lane];
        scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + wrow0 + lane] = v;
      }
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
  u64* list = list_lds[wave];
  for (int hl = wave; hl < G; hl += 4) {
    const int64_t hq = hk * G + hl;
    const float* src = scores + (b * Hq + hq) * (int64_t)nc_cap;
    int32_t* so = selected ? selected + (b * Hq + hq) * (int64_t)k : nullptr;
    float* sco = sel_scores ? sel_scores + (b * Hq + hq) * (int64_t)k : nullptr;
    int* row = sel_lds + hl * k_eff;
    if (npl <= 1) head_topk<1>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 2) head_topk<2>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 4) head_topk<4>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 8) head_topk<8>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else if (npl <= 16) head_topk<16>(src, n_cand, k, k_eff, row, so, sco, lane, list);
    else head_topk<32>(src, n_cand, k, k_eff, row, so, sco, lane, list);
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
    int Hq, int Hkv, int64_t cap, SeqArgs sa, int nc_cap, float qscale, int with_rest) {
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
  const Span sp = seq_span(sa, b);
  // item n_cand (with_rest): the tokens in no candidate segment, the window
  // and the sinks, whose mass every selection keeps
  if (s > sp.n_cand || (s == sp.n_cand && !with_rest)) return;  // wave-uniform
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

  // rows [row0, row0 + len) after the pair's base, 1 <= len <= 64: an
  // online log-sum-exp in base 2 across the tiles
  auto tile = [&](int64_t row0, int len) {
    const T* kbase = K + (bh * cap + row0) * D + jj * EPL;
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
  };
  if (s < sp.n_cand) {
    for (int off = 0; off < c; off += kTile) tile((int64_t)s * c + off, min(kTile, c - off));
  } else {
    for (int64_t st = sp.ws; st < sp.t; st += kTile) tile(st, (int)min((int64_t)kTile, sp.t - st));
    for (int off = 0; off < sp.sink; off += kTile)
      tile((int64_t)off - sa.n_sink, min(kTile, sp.sink - off));
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
      scores[(b * Hq + hk * G + g) * (int64_t)nc_cap + s] =
          l[g] > 0.f ? (m[g] + __log2f(l[g])) * kLn2 : -INFINITY;
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
  // above n = 512 the waves of a workgroup split a batch's chunks, two
  // chunks each (the four features per lane at G = 4 keep two in flight)
  constexpr int FPL = N / 64;
  constexpr int NCH = FPL <= 8 ? 1 : FPL / (G >= 4 ? 4 : 8);
  constexpr int S = NCH >= 4 ? NCH / 2 : 1;
  if constexpr (S > 1) {
    const dim3 grid((unsigned)ceil_div(n_cand, 16), (unsigned)(s.B * s.Hkv));
    const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);
    launch(RADAR_K_SCORE, k_score<N, G, S>, grid, dim3(64 * S), 0, st, phiq, summ, scores,
           s.Hq, s.Hkv, sa, s.s_cap, nc_cap);
  } else {
    constexpr int rows_per_wave = 16 * (N <= 256 ? 2 : 1);
    // waves per workgroup: 4 when that still gives two workgroups per CU,
    // else fewer, so that the rows spread over more CUs
    int wpb = 4;
    while (wpb > 1 && ceil_div(n_cand, rows_per_wave * wpb) * s.B * s.Hkv < 2 * num_cu())
      wpb >>= 1;
    const dim3 grid((unsigned)ceil_div(n_cand, rows_per_wave * wpb), (unsigned)(s.B * s.Hkv));
    const int nc_cap = (int)std::max<int64_t>(1, s.s_cap);
    launch(RADAR_K_SCORE, k_score<N, G, 1>, grid, dim3(64 * wpb), 0, st, phiq, summ, scores,
           s.Hq, s.Hkv, sa, s.s_cap, nc_cap);
  }
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
                           int n_cand, const SeqArgs& sa, int nc_cap, bool with_rest,
                           hipStream_t st) {
  const int items = n_cand + (with_rest ? 1 : 0);
  const dim3 grid((unsigned)ceil_div(items, 4), (unsigned)(s.B * s.Hkv));
  const float qscale = kLog2e / std::sqrt((float)s.d);
  const T* qt = reinterpret_cast<const T*>(q);
  const T* Kt = reinterpret_cast<const T*>(K);
  const int wr = with_rest ? 1 : 0;
  switch (s.G) {
    case 1: launch(RADAR_K_SCORE, k_segment_mass<T, D, 1>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale, wr); break;
    case 2: launch(RADAR_K_SCORE, k_segment_mass<T, D, 2>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale, wr); break;
    case 4: launch(RADAR_K_SCORE, k_segment_mass<T, D, 4>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale, wr); break;
    default: launch(RADAR_K_SCORE, k_segment_mass<T, D, 8>, grid, dim3(256), 0, st, qt, Kt, scores, s.Hq, s.Hkv, s.cap, sa, nc_cap, qscale, wr); break;
  }
}
// ---- entry points for the other units ---------------------------------------
void launch_phi_q_any(const Shape& s, const void* q, const void* omega, float* phiq,
                      hipStream_t st) {
  if (s.dt == RADAR_BF16) {
    if (s.d == 64) launch_phi_q<bf16_t, 64>(s, q, omega, phiq, st);
    else launch_phi_q<bf16_t, 128>(s, q, omega, phiq, st);
  } else {
    if (s.d == 64) launch_phi_q<float, 64>(s, q, omega, phiq, st);
    else launch_phi_q<float, 128>(s, q, omega, phiq, st);
  }
}

void launch_segment_mass(const Shape& s, const void* q, const void* K, float* scores,
                         int n_cand, const SeqArgs& sa, int nc_cap, bool with_rest,
                         hipStream_t st) {
  if (s.dt == RADAR_BF16) {
    if (s.d == 64) launch_segment_mass_d<bf16_t, 64>(s, q, K, scores, n_cand, sa, nc_cap, with_rest, st);
    else launch_segment_mass_d<bf16_t, 128>(s, q, K, scores, n_cand, sa, nc_cap, with_rest, st);
  } else {
    if (s.d == 64) launch_segment_mass_d<float, 64>(s, q, K, scores, n_cand, sa, nc_cap, with_rest, st);
    else launch_segment_mass_d<float, 128>(s, q, K, scores, n_cand, sa, nc_cap, with_rest, st);
  }
}

void launch_topk_union(const Shape& s, const float* scores, const SeqArgs& sa,
                       int* uni, int* ucnt, int umax, int32_t* selected,
                       float* sel_scores, const AppendArgs& ap, hipStream_t st) {
  launch(RADAR_K_TOPK, k_topk_union, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0, st,
         scores, s.Hq, s.Hkv, s.G, sa, (int)std::max<int64_t>(1, s.s_cap), s.per_head,
         uni, ucnt, umax, selected, sel_scores, ap, s.cap);
}

void launch_union_given(const Shape& s, const int32_t* given, int given_k,
                        const SeqArgs& sa, int* uni, int* ucnt, int umax,
                        hipStream_t st) {
  launch(RADAR_K_TOPK, k_union_given, dim3((unsigned)(s.B * s.Hkv)), dim3(256), 0, st,
         given, given_k, s.Hq, s.Hkv, s.G, sa, s.per_head, uni, ucnt, umax);
}

void launch_combine_any(const Shape& s, const float* part, const int* ucnt, void* out,
                        const SeqArgs& sa, const WsLayout& L, int tpw, int fixed_nwg,
                        int partials_per_head, hipStream_t st) {
  if (s.dt == RADAR_BF16) {
    if (s.d == 64)
      launch_combine<bf16_t, 64>(s, part, ucnt, out, sa, L, tpw, fixed_nwg, partials_per_head, st);
    else
      launch_combine<bf16_t, 128>(s, part, ucnt, out, sa, L, tpw, fixed_nwg, partials_per_head, st);
  } else {
    if (s.d == 64)
      launch_combine<float, 64>(s, part, ucnt, out, sa, L, tpw, fixed_nwg, partials_per_head, st);
    else
      launch_combine<float, 128>(s, part, ucnt, out, sa, L, tpw, fixed_nwg, partials_per_head, st);
  }
}

}  // namespace radar_impl

// Radar decode path on MI355X (gfx950, CDNA4): host logic and the C ABI.
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
//   k_peak_mfma, k_peak_exp, k_peak_read  measurement microkernels (matrix,
//                  exp2 and HBM read rates).
//
// Stages hand data to each other only inside a workgroup (LDS) or across
// kernel boundaries: the eight L2 caches of the chip are not coherent with
// one another, and the fences a cross-workgroup hand-off would need flush
// them.
//
// All softmax / feature exponentials are base 2 with log2(e) folded into the
// scale factors: exp(x) = exp2(x * log2(e)).
//
// Units: this file (host logic, C ABI, k_append, the measurement
// microkernels and the no-alloc scratch), build.hip (k_build), split.hip
// (the split path's kernels and k_combine), fused.hip (k_decode_fused, one
// unit per feature count), radar_impl.h (what they share).

#include <mutex>

#include "radar_impl.h"

namespace radar_impl {

thread_local char g_last_error[256] = "";
thread_local uint64_t* g_clock = nullptr;
thread_local int g_clock_max = 0;
thread_local Profiler g_prof;

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

radar_status launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return RADAR_OK;
  snprintf(g_last_error, sizeof g_last_error, "%s", hipGetErrorString(e));
  return RADAR_EHIP;
}
}  // namespace radar_impl

namespace {

using namespace radar_impl;

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

// The HBM read stream every decode kernel is bound by: one pass of
// non-temporal 16-byte loads over a buffer of n16 16-byte words, each
// workgroup over its own contiguous share, eight loads in flight per thread
// (the fastest of the shapes measured on MI355X: contiguous shares beat a
// grid-stride pass by 2-15%, and one 256-thread workgroup per CU with eight
// or sixteen loads in flight reached 7.26-7.27 TB/s over 4 GiB). The XOR of
// the words, one value per workgroup, keeps the loads alive.
constexpr int kPeakReadWgPerCu = 1;

__global__ __launch_bounds__(256) void k_peak_read(const uint4* __restrict__ src,
                                                   int64_t n16, float* __restrict__ sink) {
  __shared__ uint32_t red[4];
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t e = min(n16, (int64_t)blockIdx.x * per + per);
  int64_t i = (int64_t)blockIdx.x * per + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + 7 * (int64_t)blockDim.x < e; i += 8 * (int64_t)blockDim.x) {
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = ld_stream(src + i + j * blockDim.x);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (; i < e; i += blockDim.x) {
    const uint4 v = ld_stream(src + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = __uint_as_float(red[0] ^ red[1] ^ red[2] ^ red[3]);
}


// ---------------------------------------------------------------------------
// k_append: K[b][h][t] = k_new[b][h], V likewise (row pos[b] of sequence b
// when pos is given); one wave per (b, kv head)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_append(AppendArgs ap, int64_t cap, int Hkv) {
  append_row(ap, cap, blockIdx.x, Hkv, threadIdx.x);
}


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

// ---- fused path -------------------------------------------------------------
thread_local int g_path_override = RADAR_PATH_AUTO;

radar_status launch_fused_any(const FusedArgs& a, bool sel) {
  switch (a.s->n) {
    case 64: return launch_fused_n64(a, sel);
    case 128: return launch_fused_n128(a, sel);
    case 256: return launch_fused_n256(a, sel);
    case 512: return launch_fused_n512(a, sel);
    case 1024: return launch_fused_n1024(a, sel);
    default: return launch_fused_n2048(a, sel);
  }
}

// K and V start after the sinks. R workgroups per pair; with R > 1 their
// partials go to the workspace and k_combine merges them.
radar_status launch_fused(const Shape& s, const void* q, const void* K, const void* V,
                          const void* omega, const float* summ, const SeqArgs& sa,
                          void* out, int32_t* selected, float* sel_scores,
                          const AppendArgs& ap, int R, unsigned char* w,
                          const WsLayout& L, hipStream_t st) {
  float* part = R > 1 ? reinterpret_cast<float*>(w + L.part) : nullptr;
  // fp32 caches with d = 128 keep the split path: their tiles need more
  // registers than the fused kernel has to spare
  if (s.dt == RADAR_F32 && s.d == 128) return RADAR_EUNSUPPORTED;
  const FusedArgs a{&s, q, K, V, omega, summ, sa, out, selected, sel_scores, nullptr,
                    nullptr, 0, ap, R, part, L.maxwg, st, nullptr, 0};
  const radar_status r = launch_fused_any(a, false);
  if (r != RADAR_OK || R == 1) return r;
  launch_combine_any(s, part, nullptr, out, sa, L, 1, R, R, st);
  return launch_status();
}

// the select path's first kernel: phi(q), scores, top-k and union of each
// pair in one workgroup, the union into the workspace
radar_status launch_select(const Shape& s, const void* q, const void* omega,
                           const float* summ, const SeqArgs& sa, int32_t* selected,
                           float* sel_scores, unsigned char* w, const WsLayout& L,
                           const AppendArgs& ap, hipStream_t st) {
  const FusedArgs a{&s, q, nullptr, nullptr, omega, summ, sa, nullptr, selected,
                    sel_scores, reinterpret_cast<int*>(w + L.uni),
                    reinterpret_cast<int*>(w + L.ucnt), L.umax, ap, 1, nullptr, 0, st,
                    nullptr, 0};
  return launch_fused_any(a, true);
}

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
//  - scored: otherwise, where the fused kernel's register plan fits (G <= 4,
//    not fp32 with d = 128): the split path's chip-wide phi(q) and score
//    kernels, then the fused kernel from its top-k on, R workgroups per pair;
//  - split: the rest (G = 8, fp32 caches at d = 128 with many rows):
//    phi(q), scores and top-k as separate chip-wide kernels.
int choose_path(const Shape& s, const SeqArgs& sa) {
  const int n_cand = make_span(sa.t_max, sa).n_cand;
  const bool fits_select = s.G <= kFusedMaxG && n_cand <= kFusedMaxCand;
  const bool fits_fused = fits_select && !(s.dt == RADAR_F32 && s.d == 128);
  const bool fits_scored = s.G <= kFusedMaxG && !(s.dt == RADAR_F32 && s.d == 128);
  switch (g_path_override) {
    case RADAR_PATH_SPLIT: return RADAR_PATH_SPLIT;
    case RADAR_PATH_FUSED: return fits_fused ? RADAR_PATH_FUSED : RADAR_PATH_SPLIT;
    case RADAR_PATH_SELECT: return fits_select ? RADAR_PATH_SELECT : RADAR_PATH_SPLIT;
    case RADAR_PATH_SCORED: return fits_scored ? RADAR_PATH_SCORED : RADAR_PATH_SPLIT;
    default: break;
  }
  const bool few_rows = (int64_t)n_cand * s.n * 4 <= (384 << 10);
  if (fits_fused && ((int64_t)s.B * s.Hkv >= num_cu() ||
                     pair_bytes(s, sa) <= (256 << 10) || few_rows))
    return RADAR_PATH_FUSED;
  if (fits_select && few_rows) return RADAR_PATH_SELECT;
  // the rest: the scored path where the fused kernel's register plan fits
  // (measured 89.3 vs 90.5 us per step at 512K, 43.4 vs 47.2 us at the
  // paper's settings at 16K), the split path otherwise (G = 8, fp32 d = 128)
  if (fits_scored) return RADAR_PATH_SCORED;
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
  if (p->path == RADAR_PATH_FUSED || p->path == RADAR_PATH_SCORED) {
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
    launch_phi_q_any(s, q, omega, phiq, stream);
    launch_score(s, phiq, summaries, sc, top.n_cand, sa, stream);
  }
  if (plan.path == RADAR_PATH_SCORED) {
    float* part = plan.R > 1 ? reinterpret_cast<float*>(w + L.part) : nullptr;
    const FusedArgs a{&s, q, Kp, Vp, omega, summaries, sa, out, selected, scores,
                      nullptr, nullptr, 0, ap, plan.R, part, L.maxwg, stream, sc,
                      (int)std::max<int64_t>(1, s.s_cap)};
    const radar_status r = launch_fused_scored(a);
    if (r != RADAR_OK || plan.R == 1) return r;
    launch_combine_any(s, part, nullptr, out, sa, L, 1, plan.R, plan.R, stream);
    return launch_status();
  }
  launch_topk_union(s, sc, sa, reinterpret_cast<int*>(w + L.uni),
                    reinterpret_cast<int*>(w + L.ucnt), L.umax, selected, scores, ap,
                    stream);
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
      path != RADAR_PATH_SELECT && path != RADAR_PATH_SCORED)
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

radar_status radar_set_phase_clock(uint64_t* clocks, int32_t max_wgs) {
  if (clocks && (max_wgs < 1 || (reinterpret_cast<uintptr_t>(clocks) & 7u)))
    return RADAR_EINVAL;
  g_clock = clocks;
  g_clock_max = clocks ? max_wgs : 0;
  return RADAR_OK;
}

int64_t radar_wall_clock_khz(void) {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
    return 0;
  return khz;
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

radar_status radar_peak_read(const void* buf, size_t bytes, float* sink,
                             hipStream_t stream) {
  if (!buf || !sink || !aligned16(buf) || !aligned16(sink) || bytes < 16 || bytes % 16)
    return RADAR_EINVAL;
  // one sink value per workgroup: num_cu * kPeakReadWgPerCu <= the sink's
  // num_cu * kPeakWgPerCu * 256 floats
  const unsigned grid = (unsigned)(num_cu() * kPeakReadWgPerCu);
  hipLaunchKernelGGL(k_peak_read, dim3(grid), dim3(256), 0, stream,
                     static_cast<const uint4*>(buf), (int64_t)(bytes / 16), sink);
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
  if (top.n_cand > 0)
    launch_segment_mass(s, q, Kp, sc, top.n_cand, sa, (int)std::max<int64_t>(1, s.s_cap),
                        false, stream);
  launch_topk_union(s, sc, sa, reinterpret_cast<int*>(w + L.uni),
                    reinterpret_cast<int*>(w + L.ucnt), L.umax, selected, scores,
                    AppendArgs{}, stream);
  r = launch_status();
  if (r != RADAR_OK) return r;
  return launch_attend(s, q, Kp, Vp, ag, sa, out, w, L, stream);
}

radar_status radar_segment_mass(const radar_config* cfg, const void* q,
                                const void* K, int64_t t, const int64_t* lens,
                                float* ln_beta, hipStream_t stream) {
  if (!cfg || !q || !K || !ln_beta) return RADAR_EINVAL;
  if (!aligned16(q) || !aligned16(K) || !aligned16(ln_beta) || (lens && !aligned16(lens)))
    return RADAR_EINVAL;
  Shape s;
  radar_status r = check_cfg(cfg, &s);
  if (r != RADAR_OK) return r;
  if (t < 1 || t > s.cap) return RADAR_ECAPACITY;
  const SeqArgs sa{lens, t, s.c, s.w, s.n_sink, 1};
  const Span top = make_span(t, sa);
  if (top.n_cand > kMaxCand) return RADAR_EUNSUPPORTED;
  launch_segment_mass(s, q, after_sinks(s, K), ln_beta, top.n_cand, sa,
                      (int)(s.s_cap + 1), true, stream);
  return launch_status();
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
  launch_union_given(s, selected, k, sa, reinterpret_cast<int*>(w + L.uni),
                     reinterpret_cast<int*>(w + L.ucnt), L.umax, stream);
  r = launch_status();
  if (r != RADAR_OK) return r;
  return launch_attend(s, q, after_sinks(s, K), after_sinks(s, V), ag, sa, out, w,
                       L, stream);
}

}  // extern "C"


// HIP kernels of the PCTree per-round tree builder for gfx950 (CDNA4).
//
// A round (Alg. 1) runs B sequential Markov stages.  Stage d batches the
// frontier parents (Eq. 3): Z = 1 L_d^T + U W with U = SiLU(E[parents] + h_d),
// normalises every row (Eq. 2), keeps each parent's top-k children with path
// scores (Eq. 4) and prunes the layer to k frontier nodes (Sec. 4.1); after B
// stages the global top-N is emitted (Sec. 4.2, App. A).
//
// Every stage streams the whole head matrix W (V x r) once.  The V axis is cut
// into slices; a workgroup streams its slice through bf16/f32 MFMA with the
// parents as the 16 MFMA columns, folds each row into an online logsumexp and
// a per-lane top-k list, and publishes one (max, sum, top-k) partial per row:
// the V-wide child logits never leave the chip.  The partials of all slices
// are then merged and the stage's selection runs.
//
// Two launch forms:
//  * narrow (R * k' <= 16 frontier rows, one MFMA column block): ONE persistent
//    cooperative kernel per round.  After each stage the last workgroup to
//    arrive merges the slices, selects, writes the next frontier's head input
//    and releases the others; the last stage's selector also emits the tree.
//  * wide (more rows): per stage a head launch over (slice, column block) and a
//    per-request select launch; then an emit launch.
//
// Ordering keys are unique 64-bit integers, so every selection is exact and
// deterministic:
//   child key = ord(z)     << 30 | (2^20-1-token) << 10            (z desc, token asc)
//   node key  = ord(score) << 32 | (63-depth) << 26 | (2^20-1-token) << 6 | (63-slot)
//                                         (score desc, depth asc, token asc, slot asc)
// where ord() maps a float onto an unsigned integer of the same order (-0 -> +0).
#include "pctree.h"
#include "pctree_plan.h"

#include <math.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#define PCTREE_EMIT_MAX_N 256
#define PCTREE_MASK_MAX_N 1024

namespace pctree {

// The stage timeline (a diagnostic build, -DPCTREE_TIMELINE): thread 0 of a
// few workgroups stamps the device wall clock at the steps of every stage.
// The default build compiles every stamp away.
#ifdef PCTREE_TIMELINE
__device__ long long g_timeline[kTimelineWho][kTimelineStages][kTimelineEvents];
#define TIMELINE_STAMP(who, stage, ev)                                     \
  do {                                                                     \
    if (threadIdx.x == 0 && (stage) >= 0 && (stage) < kTimelineStages)      \
      g_timeline[(who)][(stage)][(ev)] = (long long)wall_clock64();         \
  } while (0)
#else
#define TIMELINE_STAMP(who, stage, ev) \
  do {                                 \
  } while (0)
#endif
// the first and the last streaming workgroup of the single-launch round
#define TIMELINE_SLICE(stage, ev)                                      \
  do {                                                                 \
    if (blockIdx.x == 0) TIMELINE_STAMP(1, stage, ev);                 \
    else if ((int)blockIdx.x == p.G - 1) TIMELINE_STAMP(2, stage, ev); \
  } while (0)

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;

// 2^x on the transcendental unit without the library's denormal-range fixups:
// terms that small (relative to a running maximum) do not change a sum of
// exponentials that holds a 1.
__device__ __forceinline__ float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }
constexpr float kNegBig = -3.0e38f;  // "no value yet" for running maxima

// A pointer known to address global memory.  Code that is not inlined into
// a kernel cannot tell where the plan's pointers point and would use flat
// accesses, which also count as LDS accesses for the waits on those.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(1))) T* gmem(const T* ptr) {
  return (const __attribute__((address_space(1))) T*)ptr;
}

__device__ __forceinline__ void __atomic_thread_fence_agent_acquire() {
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

__device__ __forceinline__ uint32_t f32_ord(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float f32_unord(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// Child keys leave their two top bits clear: read as an IEEE double, every
// key is non-negative, finite and (but 0) normal, and double order is key
// order, so the lists compare and swap them with v_max_f64 / v_min_f64.
__device__ __forceinline__ uint64_t child_key(float z, int tok) {
  return ((uint64_t)f32_ord(z) << 30) | ((uint64_t)(0xFFFFF - tok) << 10);
}

__device__ __forceinline__ int child_key_token(uint64_t key) {
  return 0xFFFFF - (int)((key >> 10) & 0xFFFFF);
}

__device__ __forceinline__ float child_key_value(uint64_t key) {
  return f32_unord((uint32_t)(key >> 30));
}

__device__ __forceinline__ uint64_t node_key(float score, int depth, int tok, int slot) {
  return ((uint64_t)f32_ord(score) << 32) | ((uint64_t)(63 - depth) << 26) |
         ((uint64_t)(0xFFFFF - tok) << 6) | (uint64_t)(63 - slot);
}

// Head input u = SiLU(E[p] + h_d): evaluated in float64 and rounded to
// nearest-even onto float32 (and then onto bf16 by the caller for a bf16 head).
__device__ __forceinline__ float silu_f32(float e, float h) {
  const double x = (double)e + (double)h;
  const double y = x / (1.0 + exp(-x));
  return (float)y;
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

// The same bf16 head input, bf16(f32(SiLU(e + h) in float64)), mostly from
// an f32 evaluation: x = e + h with its exact rounding error (two-sum),
// exp(-x) by Cody and Waite's additive range reduction (x - n ln 2 with ln 2
// split into a short high part, exact in the product, and a low part) and
// the hardware 2^x on the reduced argument, the quotient
// x / (1 + exp(-x)) refined by one Newton step, and a first-order correction
// for the rounding of x.  The result lies within 6 bit steps of
// f32(SiLU64(x)) by the error analysis (at most 3 seen over 10^9 draws with
// |x| from 1e-3 to 30), so it rounds to the same bf16 unless it lies within
// kSiluTol steps of a bf16 rounding midpoint.  Those elements (about 1 in
// 4000), |x| >= 16, and zero or subnormal results take the float64 path.
constexpr int kSiluTol = 8;
__device__ __forceinline__ uint16_t silu_bf16(float e, float h) {
  const float x = e + h;
  const float bb = x - e;
  const float xe = (e - (x - bb)) + (h - bb);  // x + xe == e + h exactly
  const float n = rintf(-x * kLog2e);
  float r = fmaf(n, -0.693145751953125f, -x);  // ln 2 split: 0x3f317200 + 0x35bfbe8e
  r = fmaf(n, -1.428606820309417232e-06f, r);
  const float t = __builtin_amdgcn_ldexpf(exp2_raw(r * kLog2e), (int)n);  // exp(-x)
  const float d = 1.0f + t;
  float q = __builtin_amdgcn_rcpf(d);
  q = fmaf(q, fmaf(-d, q, 1.0f), q);
  float y = x * q;
  y = fmaf(fmaf(-y, d, x), q, y);
  y = fmaf(q * fmaf(x * t, q, 1.0f), xe, y);  // + SiLU'(x) * xe
  const uint32_t b = __float_as_uint(y);
  const int lo = (int)(b & 0xffffu) - 0x8000;
  const bool ok = fabsf(x) < 16.0f && (lo > kSiluTol || lo < -kSiluTol) && (b & 0x7f800000u) != 0u;
  return bf16_rne(ok ? y : silu_f32(e, h));
}

template <int DT>
__device__ __forceinline__ float load_elem(const void* base, size_t i) {
  if (DT) return __uint_as_float((uint32_t)((const uint16_t*)base)[i] << 16);
  return ((const float*)base)[i];
}

// Selection state of a round: the frontier (slot-indexed, kk per request) and
// the running global top-N (sorted keys and pool ids, N per request).  It
// lives in the workspace for the multi-launch form and in the selector
// workgroup's LDS for the persistent form.
// Entry i of request req sits at [(req - rbase) * kk + slot] (frontier) and
// [(req - rbase) * N + i] (top-N): rbase 0 for state holding every request,
// req for a copy of one request's.
struct State {
  int* front_node;
  int* front_tok;
  float* front_score;
  uint64_t* top_key;
  int* top_node;
  int rbase;
};

__device__ __forceinline__ State global_state(const Plan& p) {
  return State{p.front_node, p.front_tok, p.front_score, p.top_key, p.top_node, 0};
}

// ---------------------------------------------------------------------------
// sorted (descending) fixed-length candidate lists held in registers
// ---------------------------------------------------------------------------
// Larger / smaller of two child keys (see child_key) on the double ALU.
__device__ __forceinline__ uint64_t key_max(uint64_t a, uint64_t b) {
  return (uint64_t)__double_as_longlong(
      __builtin_fmax(__longlong_as_double((long long)a), __longlong_as_double((long long)b)));
}
__device__ __forceinline__ uint64_t key_min(uint64_t a, uint64_t b) {
  return (uint64_t)__double_as_longlong(
      __builtin_fmin(__longlong_as_double((long long)a), __longlong_as_double((long long)b)));
}

template <int K>
__device__ __forceinline__ void list_insert(uint64_t (&l)[K], uint64_t key) {
  l[K - 1] = key;
#pragma unroll
  for (int i = K - 1; i > 0; --i) {
    const uint64_t a = l[i - 1], b = l[i];
    l[i - 1] = key_max(a, b);
    l[i] = key_min(a, b);
  }
}

// a <- top-K of (a u b); both sorted descending.  Elementwise max against the
// reversed b gives a bitonic sequence holding the top K; half-cleaners sort it.
template <int K>
__device__ __forceinline__ void list_merge(uint64_t (&a)[K], const uint64_t (&b)[K]) {
#pragma unroll
  for (int i = 0; i < K; ++i) a[i] = key_max(a[i], b[K - 1 - i]);
#pragma unroll
  for (int j = K / 2; j > 0; j >>= 1) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if ((i & j) == 0) {
        const uint64_t x = a[i], y = a[i + j];
        a[i] = key_max(x, y);
        a[i + j] = key_min(x, y);
      }
    }
  }
}

// a <- top-K of (a u n), n four keys sorted descending (K >= 4): only the
// last four entries of a can give way, then half-cleaners sort the result.
template <int K>
__device__ __forceinline__ void list_merge4(uint64_t (&a)[K], const uint64_t (&n)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) a[K - 4 + i] = key_max(a[K - 4 + i], n[3 - i]);
#pragma unroll
  for (int j = K / 2; j > 0; j >>= 1) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if ((i & j) == 0) {
        const uint64_t x = a[i], y = a[i + j];
        a[i] = key_max(x, y);
        a[i + j] = key_min(x, y);
      }
    }
  }
}

template <int K>
__device__ __forceinline__ void list_merge_xor(uint64_t (&l)[K], int mask) {
  uint64_t o[K];
#pragma unroll
  for (int i = 0; i < K; ++i) o[i] = __shfl_xor(l[i], mask);
  list_merge(l, o);
}

// Exchange with lane ^ 16 / lane ^ 32 on the VALU (v_permlane{16,32}_swap):
// each returns {own, partner} in a lane-dependent order, which a symmetric
// combine (list merge, lse combine) does not care about.
template <int X>
__device__ __forceinline__ void swap_pair(uint32_t v, uint32_t& a, uint32_t& b) {
  if constexpr (X == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    a = r[0];
    b = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    a = r[0];
    b = r[1];
  }
}

template <int X, int K>
__device__ __forceinline__ void list_merge_pair(uint64_t (&l)[K]) {
  uint64_t a[K], b[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    uint32_t alo, blo, ahi, bhi;
    swap_pair<X>((uint32_t)l[i], alo, blo);
    swap_pair<X>((uint32_t)(l[i] >> 32), ahi, bhi);
    a[i] = ((uint64_t)ahi << 32) | alo;
    b[i] = ((uint64_t)bhi << 32) | blo;
  }
  list_merge(a, b);
#pragma unroll
  for (int i = 0; i < K; ++i) l[i] = a[i];
}

// Wave-wide reductions on DPP lane permutations (VALU latency, not the LDS
// path of a shuffle): within each 16-lane row by quad permutes and mirrors,
// then across rows by broadcasts of lanes 15 and 31; lane 63 ends with the
// result, which is read back into a uniform value.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false);
}

template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  return ((uint64_t)dpp<CTRL, ROWS>((uint32_t)(v >> 32)) << 32) | dpp<CTRL, ROWS>((uint32_t)v);
}

__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// Keys are >= 0, so 0 (what DPP yields for lanes outside the row mask) is
// the identity of the maximum.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp<0xB1, 0xF>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp<0x4E, 0xF>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp<0x141, 0xF>(v));  // row_half_mirror
  v = max(v, dpp<0x140, 0xF>(v));  // row_mirror
  v = max(v, dpp<0x142, 0xA>(v));  // row_bcast15 into rows 1, 3
  v = max(v, dpp<0x143, 0xC>(v));  // row_bcast31 into rows 2, 3
  return __builtin_amdgcn_readlane(v, 63);
}

// The maximum over the wave of a u64 key: the high words decide; the low word
// comes from the one lane holding the maximal high word, or from a second
// reduction over the tied lanes.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  const uint32_t hi = (uint32_t)(v >> 32);
  const uint32_t lo = (uint32_t)v;
  const uint32_t mh = wave_max_u32(hi);
  const uint64_t tied = __ballot(hi == mh);
  uint32_t ml;
  if ((tied & (tied - 1)) == 0)
    ml = __builtin_amdgcn_readlane(lo, __builtin_ctzll(tied));
  else
    ml = wave_max_u32(hi == mh ? lo : 0u);
  return ((uint64_t)mh << 32) | ml;
}

template <int CTRL, int ROWS>
__device__ __forceinline__ float dppf(float v, float identity) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_update_dpp(
      (int)__float_as_uint(identity), (int)__float_as_uint(v), CTRL, ROWS, 0xF, false));
}

__device__ __forceinline__ float wave_max_f32(float v) {
  v = fmaxf(v, dppf<0xB1, 0xF>(v, kNegBig));
  v = fmaxf(v, dppf<0x4E, 0xF>(v, kNegBig));
  v = fmaxf(v, dppf<0x141, 0xF>(v, kNegBig));
  v = fmaxf(v, dppf<0x140, 0xF>(v, kNegBig));
  v = fmaxf(v, dppf<0x142, 0xA>(v, kNegBig));
  v = fmaxf(v, dppf<0x143, 0xC>(v, kNegBig));
  return __uint_as_float(__builtin_amdgcn_readlane((int)__float_as_uint(v), 63));
}

__device__ __forceinline__ float wave_sum_f32(float v) {
  v += dppf<0xB1, 0xF>(v, 0.0f);
  v += dppf<0x4E, 0xF>(v, 0.0f);
  v += dppf<0x141, 0xF>(v, 0.0f);
  v += dppf<0x140, 0xF>(v, 0.0f);
  v += dppf<0x142, 0xA>(v, 0.0f);
  v += dppf<0x143, 0xC>(v, 0.0f);
  return __uint_as_float(__builtin_amdgcn_readlane((int)__float_as_uint(v), 63));
}

// (m, s) pairs describe sum_i exp(z_i) = exp(m) * s; combine two of them.
__device__ __forceinline__ void lse_combine(float& m, float& s, float om, float os) {
  const float nm = fmaxf(m, om);
  s = s * exp2_raw((m - nm) * kLog2e) + os * exp2_raw((om - nm) * kLog2e);
  m = nm;
}

__device__ __forceinline__ void lse_combine_xor(float& m, float& s, int mask) {
  const float om = __shfl_xor(m, mask);
  const float os = __shfl_xor(s, mask);
  lse_combine(m, s, om, os);
}

template <int X>
__device__ __forceinline__ void lse_combine_pair(float& m, float& s) {
  uint32_t m0, m1, s0, s1;
  swap_pair<X>(__float_as_uint(m), m0, m1);
  swap_pair<X>(__float_as_uint(s), s0, s1);
  m = __uint_as_float(m0);
  s = __uint_as_float(s0);
  lse_combine(m, s, __uint_as_float(m1), __uint_as_float(s1));
}

// ---------------------------------------------------------------------------
// MFMA on one 16-byte rank chunk per lane
// ---------------------------------------------------------------------------
template <int DT>
__device__ __forceinline__ f32x4 mfma_chunk(u32x4 a, u32x4 b, f32x4 acc);

template <>
__device__ __forceinline__ f32x4 mfma_chunk<1>(u32x4 a, u32x4 b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x4 mfma_chunk<0>(u32x4 a, u32x4 b, f32x4 acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[i]), __uint_as_float(b[i]), acc,
                                               0, 0, 0);
  return acc;
}

// ---------------------------------------------------------------------------
// prologue: root node, frontier {x_t}, running top-N {root}, head input of x_t
// ---------------------------------------------------------------------------
// Per-request outputs and pool entries every form starts from: the root node
// (token 0 stands in for an invalid root, whose tree is emitted empty), a
// count of -1 that stays if the round is aborted, the trace's stage-0 row.
// Threads [tid0, tid0 + nth) of the calling workgroup share the work.
__device__ __forceinline__ void init_request_body(const Plan& p, int req, int tid, int nth) {
  int root = p.root[req];
  const bool bad = root < 0 || root >= p.V;
  if (bad) root = 0;
  if (tid == 0) {
    p.req_bad[req] = bad ? 1 : 0;
    p.o_count[req] = -1;
    const size_t nb = (size_t)req * p.maxpool;
    p.node_tok[nb] = root;
    p.node_par[nb] = -1;
    p.node_depth[nb] = 0;
    p.node_score[nb] = 0.0f;
  }
  if (p.t_token) {
    const int n = p.B * p.k;
    for (int i = tid; i < n; i += nth) {
      const size_t o = (size_t)req * n + i;
      const bool first = i == 0;
      p.t_token[o] = first ? root : -1;
      p.t_pslot[o] = -1;
      p.t_score[o] = first ? 0.0f : -INFINITY;
    }
  }
}

__device__ void init_request(const Plan& p, int req, int tid, int nth) {
  init_request_body(p, req, tid, nth);
}

// Head rows per request of stage d, and whether stage d of a per-stage-launch
// round runs the wide form: when it has more than 16 head rows, and in every
// stage of a round whose frontier can exceed 16 rows (the stages with fewer
// rows then also take the bounded head stream and the one merge-and-select
// launch: 900 -> 893 us per round at 8 requests with k' = 16, and 867 -> 820
// and 849 -> 794 us in the two control scorings, whose stages all have one
// row per request).  Rounds with at most 16 frontier rows launched per stage
// keep the narrow form.
__device__ __host__ __forceinline__ int head_rows(int mode, int d, int kk) {
  return (d == 0 || mode != 0) ? 1 : kk;
}
__device__ __host__ __forceinline__ bool stage_wide(int mode, int d, int R, int kk) {
  return R * head_rows(mode, d, kk) > kNarrowRows || R * kk > kNarrowRows;
}

// ---------------------------------------------------------------------------
// head stream over one V-slice for one block of 16 frontier rows
// ---------------------------------------------------------------------------
// MFMA 16x16xK with tokens as M and frontier rows as N: lane l feeds A row
// (token) l%16 and B column (row) l%16 with rank chunk group l/16, and
// receives C[token 4*(l/16)+i][row l%16], i = 0..3.
template <int KMAX, int WAVES>
struct HeadShared {
  // key-major, so that the 16 or 64 lanes writing or reading key i of their
  // rows touch consecutive words (no bank conflicts)
  uint64_t wl[KMAX][WAVES][kTile];
  uint64_t wt[KMAX < 4 ? KMAX : 4][WAVES][kTile];
  float2 wms[WAVES][kTile];
};

template <int NCMAX>
struct Tile {
  u32x4 a[NCMAX];
  uint32_t l[4];  // raw bits of L_d (bf16 in the low half, or f32)
};

template <int DT>
__device__ __forceinline__ uint32_t load_raw(const void* base, size_t i) {
  if (DT) return ((const uint16_t*)base)[i];
  return ((const uint32_t*)base)[i];
}

template <int DT>
__device__ __forceinline__ float raw_to_f32(uint32_t r) {
  return __uint_as_float(DT ? r << 16 : r);
}

// Lane geometry of a head pass over one block of 16 frontier rows.
// With `fold` (at most 8 frontier rows) the C fragments of two tiles share
// the 16 columns: columns 0..7 keep the first tile's rows, columns 8..15 take
// the second tile's (moved up by 8), so that every lane holds a live row.  B
// columns (the frontier rows fed to the MFMA) are unaffected.
struct HeadLane {
  int lane, wave, col, grp;
  int row, req, slot;  // the frontier row whose logits this lane holds
  bool row_ok;
  int half;            // which tile of a folded pair (0 without fold)
  bool lead;           // the lane that publishes its row (first of a folded pair)
  int b_req, b_slot;   // the frontier row of this lane's B column
  bool b_ok;
  __device__ HeadLane(const Plan& p, int P, int cb, bool fold = false) {
    lane = threadIdx.x & 63;
    wave = threadIdx.x >> 6;
    col = lane & 15;
    grp = lane >> 4;
    const int nrows = p.R * P;
    const int bcol = cb * kTile + col;
    b_ok = bcol < nrows;
    b_req = b_ok ? bcol / P : 0;
    b_slot = b_ok ? bcol - b_req * P : 0;
    row = cb * kTile + (fold ? (col & 7) : col);
    row_ok = row < nrows;
    req = row_ok ? row / P : 0;
    slot = row_ok ? row - req * P : 0;
    half = fold ? (col >> 3) : 0;
    lead = !fold || col < 8;
  }
};

// B fragments: the head input u of this lane's frontier row.
template <int DT, int NCMAX>
__device__ __forceinline__ void load_bfrag(const Plan& p, const HeadLane& h, u32x4 (&b)[NCMAX]) {
  constexpr int KC = DT ? 32 : 16;
  constexpr int ESZ = DT ? 2 : 4;
  const char* urow =
      (const char*)p.U + ((size_t)(h.b_req * p.kk + h.b_slot) * p.r + h.grp * (KC / 4)) * ESZ;
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (c < p.nchunk && h.b_ok) v = *(const u32x4*)(urow + (size_t)c * KC * ESZ);
    b[c] = v;
  }
}

// A fragments of tile t (16 tokens x r) for this lane.  No branch: the token
// is clamped into the vocabulary (rows of tokens >= V are discarded later),
// chunks past the rank re-read the last chunk and meet zero B fragments.
template <int DT, int NCMAX>
__device__ __forceinline__ void load_afrag(const Plan& p, const HeadLane& h, int t,
                                           u32x4 (&a)[NCMAX]) {
  constexpr int KC = DT ? 32 : 16;
  constexpr int ESZ = DT ? 2 : 4;
  const int tok = min(t * kTile + h.col, p.V - 1);
  const char* wrow = (const char*)p.Wt + ((size_t)tok * p.r + h.grp * (KC / 4)) * ESZ;
#pragma unroll
  for (int c = 0; c < NCMAX; ++c)
    a[c] = *(const u32x4*)(wrow + (size_t)min(c, p.nchunk - 1) * KC * ESZ);
}

// L_d of the four tokens of tile t this lane's C fragment holds (raw bits).
template <int DT>
__device__ __forceinline__ void load_lfrag(const Plan& p, const HeadLane& h, int d, int t,
                                           uint32_t (&l)[4]) {
  const size_t lrow = ((size_t)h.req * p.B + d) * p.V;
  const int tb = t * kTile + h.grp * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) l[i] = load_raw<DT>(p.L, lrow + min(tb + i, p.V - 1));
}

// Per-lane running state of a row: online (max, sum of exp) and top-KMAX keys.
template <int KMAX>
struct RowAcc {
  float m, s;
  uint64_t list[KMAX];
  __device__ void init() {
    m = kNegBig;
    s = 0.0f;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) list[i] = 0;
  }
};

__device__ __forceinline__ void cas_desc(uint64_t& a, uint64_t& b) {
  const uint64_t hi = key_max(a, b), lo = key_min(a, b);
  a = hi;
  b = lo;
}

// The lane's four logits of tile t (C fragment + L_d), folded into its row's
// online logsumexp and top-k list when `ok`.  Four new keys enter a list of
// at least four as one sorted batch (a 4-sort, then the list merge); shorter
// lists take them one at a time.  Only the last tile of the vocabulary can
// hold tokens past V, and only there are they masked one by one.
template <int DT, int KMAX>
__device__ __forceinline__ void tile_epilogue(const Plan& p, const HeadLane& h, f32x4 acc,
                                              const uint32_t (&l)[4], int t, bool ok,
                                              RowAcc<KMAX>& r) {
  if (ok) {
    const int tb = t * kTile + h.grp * 4;
    float z[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) z[i] = acc[i] + raw_to_f32<DT>(l[i]);
    if (tb + 3 < p.V) {
      const float nm = fmaxf(fmaxf(r.m, fmaxf(z[0], z[1])), fmaxf(z[2], z[3]));
      float ss = r.s * exp2_raw((r.m - nm) * kLog2e);
#pragma unroll
      for (int i = 0; i < 4; ++i) ss += exp2_raw((z[i] - nm) * kLog2e);
      r.m = nm;
      r.s = ss;
      uint64_t n[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) n[i] = child_key(z[i], tb + i);
      if constexpr (KMAX >= 4) {
        cas_desc(n[0], n[1]);
        cas_desc(n[2], n[3]);
        cas_desc(n[0], n[2]);
        cas_desc(n[1], n[3]);
        cas_desc(n[1], n[2]);
        list_merge4(r.list, n);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (n[i] > r.list[KMAX - 1]) list_insert(r.list, n[i]);
      }
    } else {
      float tmax = kNegBig;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (tb + i >= p.V) z[i] = kNegBig;
        tmax = fmaxf(tmax, z[i]);
      }
      const float nm = fmaxf(r.m, tmax);
      float ss = r.s * exp2_raw((r.m - nm) * kLog2e);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (tb + i < p.V) ss += exp2_raw((z[i] - nm) * kLog2e);
      r.m = nm;
      r.s = ss;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (tb + i < p.V) {
          const uint64_t key = child_key(z[i], tb + i);
          if (key > r.list[KMAX - 1]) list_insert(r.list, key);
        }
      }
    }
  }
}

// One tile: Z = A B^T on MFMA, then the epilogue.
template <int DT, int NCMAX, int KMAX>
__device__ __forceinline__ void tile_step(const Plan& p, const HeadLane& h,
                                          const u32x4 (&a)[NCMAX], const u32x4 (&b)[NCMAX],
                                          const uint32_t (&l)[4], int t, RowAcc<KMAX>& r) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) acc = mfma_chunk<DT>(a[c], b[c], acc);
  tile_epilogue<DT, KMAX>(p, h, acc, l, t, h.row_ok, r);
}


// Two tiles on two independent MFMA chains; the second tile's C fragment is
// moved into columns 8..15 (DPP row_shr:8 onto banks 2-3 of every row), then
// one epilogue covers both.  t is the lane's own tile (ta or tb by half).
template <int DT, int NCMAX, int KMAX>
__device__ __forceinline__ void tile_pair_step(const Plan& p, const HeadLane& h,
                                               const u32x4 (&a0)[NCMAX], const u32x4 (&a1)[NCMAX],
                                               const u32x4 (&b)[NCMAX], const uint32_t (&l)[4],
                                               int t, bool ok, RowAcc<KMAX>& r) {
  f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) {
    c0 = mfma_chunk<DT>(a0[c], b[c], c0);
    c1 = mfma_chunk<DT>(a1[c], b[c], c1);
  }
  f32x4 acc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    acc[i] = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(c0[i]), __float_as_int(c1[i]),
                                                        0x118, 0xF, 0xC, false));
  tile_epilogue<DT, KMAX>(p, h, acc, l, t, ok && h.row_ok, r);
}

// tile_pair_step on two LDS-resident tiles (fragment order), reading each
// rank chunk right before its MFMA so that only two chunks are live.
template <int DT, int NCMAX, int KMAX>
__device__ __forceinline__ void lds_pair_step(const Plan& p, const HeadLane& h, const u32x4* w0,
                                              const u32x4* w1, const u32x4 (&b)[NCMAX],
                                              const uint32_t (&l)[4], int t, bool ok,
                                              RowAcc<KMAX>& r) {
  f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) {
    c0 = mfma_chunk<DT>(w0[c * 64], b[c], c0);
    c1 = mfma_chunk<DT>(w1[c * 64], b[c], c1);
  }
  f32x4 acc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    acc[i] = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(c0[i]), __float_as_int(c1[i]),
                                                        0x118, 0xF, 0xC, false));
  tile_epilogue<DT, KMAX>(p, h, acc, l, t, ok && h.row_ok, r);
}

// Word 0 of slice 0 of the (stage, row) slice records; word w of slice s is
// at + w * kSlicesMax + s.
__device__ __forceinline__ uint64_t* slice_record(const Plan& p, int stage, int row) {
  return p.part_hd + ((size_t)stage * p.rows_max + row) * kRecWords * kSlicesMax;
}

// Reduce the lanes' row states over the workgroup and publish the slice's
// partial of every row.  Two reduction trees: the first carries only the
// lanes' best four keys and the (max, sum) pairs and ends in the record, which
// is all the keeper needs unless a row's record keys do not settle it; the
// second then carries the full lists, which only that rare case reads.
// Rows live in lanes col, col+16, col+32, col+48 of every wave (and, folded,
// in lanes col and col ^ 8).
template <int KMAX, int WAVES, bool FOLD = false>
__device__ __forceinline__ void publish_partial(const Plan& p, const HeadLane& h, int stage,
                                                int slice, RowAcc<KMAX>& r,
                                                HeadShared<KMAX, WAVES>& sh) {
  constexpr int HT = KMAX < 4 ? KMAX : 4;
  const size_t o = ((size_t)stage * p.rows_max + h.row) * kSlicesMax + slice;
  const bool writer = h.grp == 0 && h.row_ok && h.lead;
  {
    uint64_t t[HT];
#pragma unroll
    for (int i = 0; i < HT; ++i) t[i] = r.list[i];
    float m = r.m, sum = r.s;
    if constexpr (FOLD) {
      uint64_t x[HT];
#pragma unroll
      for (int i = 0; i < HT; ++i) x[i] = dpp64<0x128, 0xF>(t[i]);
      list_merge(t, x);
      lse_combine(m, sum, dppf<0x128, 0xF>(m, kNegBig), dppf<0x128, 0xF>(sum, 0.0f));
    }
    list_merge_pair<16>(t);
    lse_combine_pair<16>(m, sum);
    list_merge_pair<32>(t);
    lse_combine_pair<32>(m, sum);
    if (h.grp == 0) {
#pragma unroll
      for (int i = 0; i < HT; ++i) sh.wt[i][h.wave][h.col] = t[i];
      sh.wms[h.wave][h.col] = make_float2(m, sum);
    }
    __syncthreads();
    if (h.wave == 0) {
#pragma unroll
      for (int i = 0; i < HT; ++i) t[i] = sh.wt[i][h.grp][h.col];
      m = sh.wms[h.grp][h.col].x;
      sum = sh.wms[h.grp][h.col].y;
#pragma unroll
      for (int w = h.grp + 4; w < WAVES; w += 4) {
        uint64_t x[HT];
#pragma unroll
        for (int i = 0; i < HT; ++i) x[i] = sh.wt[i][w][h.col];
        list_merge(t, x);
        lse_combine(m, sum, sh.wms[w][h.col].x, sh.wms[w][h.col].y);
      }
      list_merge_pair<16>(t);
      lse_combine_pair<16>(m, sum);
      list_merge_pair<32>(t);
      lse_combine_pair<32>(m, sum);
      if (writer) {
        // tagged words, stored write-through at agent scope: each one is
        // valid on its own once it lands (keys have their low kTagBits clear)
        uint64_t* hd = slice_record(p, stage, h.row) + slice;
#pragma unroll
        for (int i = 0; i < kHeadKeys; ++i)
          __hip_atomic_store(hd + i * kSlicesMax, (i < HT ? t[i < HT ? i : 0] : 0ull) | p.tag,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // the sum relative to the best logit (m is the logit of t[0])
        __hip_atomic_store(hd + kHeadKeys * kSlicesMax,
                           ((uint64_t)p.tag << 32) | __float_as_uint(sum), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (HT == KMAX) {
          uint64_t* dst = p.part_key + o * KMAX;
#pragma unroll
          for (int i = 0; i < KMAX; ++i)
            __hip_atomic_store(dst + i, t[i] | p.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }
  if constexpr (HT < KMAX) {
    if constexpr (FOLD) {
      uint64_t x[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) x[i] = dpp64<0x128, 0xF>(r.list[i]);
      list_merge(r.list, x);
    }
    list_merge_pair<16>(r.list);
    list_merge_pair<32>(r.list);
    if (h.grp == 0) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) sh.wl[i][h.wave][h.col] = r.list[i];
    }
    __syncthreads();
    if (h.wave == 0) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) r.list[i] = sh.wl[i][h.grp][h.col];
#pragma unroll
      for (int w = h.grp + 4; w < WAVES; w += 4) {
        uint64_t x[KMAX];
#pragma unroll
        for (int i = 0; i < KMAX; ++i) x[i] = sh.wl[i][w][h.col];
        list_merge(r.list, x);
      }
      list_merge_pair<16>(r.list);
      list_merge_pair<32>(r.list);
      if (writer) {
        uint64_t* dst = p.part_key + o * KMAX;
#pragma unroll
        for (int i = 0; i < KMAX; ++i)
          __hip_atomic_store(dst + i, r.list[i] | p.tag, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Published words of this call (see kTagBits).
__device__ __forceinline__ bool key_tagged(const Plan& p, uint64_t w) {
  return ((uint32_t)w & kTagMask) == p.tag;
}
__device__ __forceinline__ bool sum_tagged(const Plan& p, uint64_t w) {
  return (uint32_t)(w >> 32) == p.tag;
}
__device__ __forceinline__ uint64_t load_agent(const uint64_t* ptr) {
  return __hip_atomic_load(ptr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Stream one slice of W for one block of 16 frontier rows (multi-launch form):
// the next tiles' loads are in flight while this one computes (three tiles in
// registers up to rank 256, else two).  Prefetches are unconditional (clamped
// to the slice's last tile, surplus ones are never processed) so that the
// compiler's waits on the loads in flight stay partial.
template <int DT, int NCMAX, int KMAX, int WAVES>
__device__ __forceinline__ void head_slice(const Plan& p, int d, int P, int cb, int slice,
                                           HeadShared<KMAX, WAVES>& sh) {
  const HeadLane h(p, P, cb);
  u32x4 bfrag[NCMAX];
  load_bfrag<DT, NCMAX>(p, h, bfrag);
  RowAcc<KMAX> r;
  r.init();
  auto load = [&](Tile<NCMAX>& T, int t) {
    load_afrag<DT, NCMAX>(p, h, t, T.a);
    load_lfrag<DT>(p, h, d, t, T.l);
  };
  auto process = [&](const Tile<NCMAX>& T, int t) {
    tile_step<DT, NCMAX, KMAX>(p, h, T.a, bfrag, T.l, t, r);
  };
  const int t1 = min((slice + 1) * p.tiles_per_slice, p.ntiles);
  int t = slice * p.tiles_per_slice + h.wave;
  Tile<NCMAX> TA, TB;
  load(TA, min(t, t1 - 1));
  if constexpr (NCMAX <= 8) {
    Tile<NCMAX> TC;
    load(TB, min(t + WAVES, t1 - 1));
    while (t < t1) {
      load(TC, min(t + 2 * WAVES, t1 - 1));
      process(TA, t);
      t += WAVES;
      if (t >= t1) break;
      load(TA, min(t + 2 * WAVES, t1 - 1));
      process(TB, t);
      t += WAVES;
      if (t >= t1) break;
      load(TB, min(t + 2 * WAVES, t1 - 1));
      process(TC, t);
      t += WAVES;
    }
  } else {
    while (t < t1) {
      load(TB, min(t + WAVES, t1 - 1));
      process(TA, t);
      t += WAVES;
      if (t >= t1) break;
      load(TA, min(t + WAVES, t1 - 1));
      process(TB, t);
      t += WAVES;
    }
  }
  publish_partial<KMAX, WAVES>(p, h, 0, slice, r, sh);
}

// Tiles a streaming block of the persistent kernel keeps on chip for the
// whole round: RT per wave in registers and up to LTW per wave in LDS.
// (64 VGPRs of resident A fragments per lane at most: more spills.)
__host__ __device__ constexpr int resident_reg_tiles(int ncmax, bool fold = false) {
  if (fold) return ncmax <= 2 ? 4 : (ncmax <= 4 ? 3 : (ncmax <= 8 ? 3 : 1));
  return ncmax <= 2 ? 4 : (ncmax <= 4 ? 3 : (ncmax <= 8 ? 2 : 1));
}
__host__ __device__ constexpr int resident_lds_tiles_per_wave(int ncmax) {
  return ncmax <= 4 ? 4 : (ncmax <= 8 ? 2 : 1);
}

// A streaming block of the persistent kernel.  W of its slice is read from
// memory once per round: the first RT*WAVES tiles go to registers, the next
// p.lds_tiles to LDS (stored in MFMA fragment order), and only the rest, if
// any, is streamed at every stage.  Each stage then loads L_d before waiting
// for the selector's release, reads the new head input and runs the tiles.
// ---------------------------------------------------------------------------
// persistent form: replicated selection
// ---------------------------------------------------------------------------
// Every workgroup keeps its own copy of the frontier (identical everywhere:
// all derive it from the same published partials with the same code).
struct FrontShared {
  int tok[kNarrowRows];
  float score[kNarrowRows];
};

// Head input of the frontier in LDS: [rows][r] at the head's precision, rows
// padded by 16 bytes so that the 16 columns' B-fragment reads spread over
// the banks.
__device__ __forceinline__ int u_stride(const Plan& p) { return p.r * (p.dtype ? 2 : 4) + 16; }

template <int DT>
__device__ void compute_u(const Plan& p, const FrontShared& fs, int d, int P, char* ul) {
  constexpr int Q = 4;  // elements per work item
  const int rows = p.R * P;
  const int us = u_stride(p);
  const int n = rows * p.r / Q;
  for (int base = 0; base < n; base += 2 * (int)blockDim.x) {
    uint32_t ev[2][Q];
    f32x4 hv[2];
    int urow[2], j0[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = min(base + q * (int)blockDim.x + (int)threadIdx.x, n - 1) * Q;
      const int row = e / p.r;
      const int j = e - row * p.r;
      const int req = row / P;
      const int tok = min(max(fs.tok[req * p.kk + (row - req * P)], 0), p.V - 1);
      const size_t eo = (size_t)tok * p.r + j;
      if (DT) {
        const u32x2 v = *gmem((const u32x2*)((const uint16_t*)p.E + eo));
        ev[q][0] = v.x << 16;
        ev[q][1] = v.x & 0xffff0000u;
        ev[q][2] = v.y << 16;
        ev[q][3] = v.y & 0xffff0000u;
      } else {
        const u32x4 v = *gmem((const u32x4*)((const float*)p.E + eo));
#pragma unroll
        for (int i = 0; i < Q; ++i) ev[q][i] = v[i];
      }
      hv[q] = *gmem((const f32x4*)(p.h + ((size_t)req * p.B + d) * p.r + j));
      urow[q] = row;
      j0[q] = j;
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (base + q * (int)blockDim.x + (int)threadIdx.x < n) {
        char* dst = ul + (size_t)urow[q] * us;
        if (p.mode == 2) {  // parent-independent: zero head input
          if (DT)
            *(uint2*)(dst + j0[q] * 2) = uint2{0u, 0u};
          else
            *(f32x4*)(dst + j0[q] * 4) = f32x4{0.f, 0.f, 0.f, 0.f};
        } else if (DT) {
          uint16_t u[Q];
#pragma unroll
          for (int i = 0; i < Q; ++i) u[i] = silu_bf16(__uint_as_float(ev[q][i]), hv[q][i]);
          uint2 v;
          v.x = (uint32_t)u[0] | ((uint32_t)u[1] << 16);
          v.y = (uint32_t)u[2] | ((uint32_t)u[3] << 16);
          *(uint2*)(dst + j0[q] * 2) = v;
        } else {
          float u[Q];
#pragma unroll
          for (int i = 0; i < Q; ++i) u[i] = silu_f32(__uint_as_float(ev[q][i]), hv[q][i]);
          *(f32x4*)(dst + j0[q] * 4) = f32x4{u[0], u[1], u[2], u[3]};
        }
      }
    }
  }
  __syncthreads();
}

// B fragments from the head input in LDS (zero past the rows and the rank).
template <int DT, int NCMAX>
__device__ __forceinline__ void load_bfrag_lds(const Plan& p, const HeadLane& h, const char* ul,
                                               u32x4 (&b)[NCMAX]) {
  constexpr int KC = DT ? 32 : 16;
  constexpr int ESZ = DT ? 2 : 4;
  const char* urow = ul + (size_t)h.col * u_stride(p) + h.grp * (KC / 4) * ESZ;
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (c < p.nchunk && h.b_ok) v = *(const u32x4*)(urow + c * KC * ESZ);
    b[c] = v;
  }
}


template <int DT>
__device__ __noinline__ void frontier_call(const Plan& lp, int d);

// Wave 0 waits for the stage-d frontier that the keeper publishes (R*k'
// words, each carrying the call's tag: score bits << 32 | token << kTagBits
// | tag) and puts its tokens into fs.  Polls with agent-coherent loads,
// bounded by p.spin_ticks of the device wall clock: returns 0 on a timeout.
__device__ __forceinline__ int wait_frontier(const Plan& p, int d, FrontShared& fs) {
  const int lane = threadIdx.x & 63;
  const int n = p.R * p.kk;  // <= kNarrowRows
  const uint64_t* src = p.front_w + (size_t)d * p.rows_max + min(lane, n - 1);
  const long long t0 = wall_clock64();
  uint64_t w;
  for (;;) {
    w = load_agent(src);
    if (__all(key_tagged(p, w))) break;
    if (wall_clock64() - t0 > p.spin_ticks) return 0;
    __builtin_amdgcn_s_sleep(1);
  }
  if (lane < n) fs.tok[lane] = min((int)((uint32_t)w >> kTagBits), p.V - 1);
  return 1;
}

// Everything a streaming workgroup does before its stage-d stream: wait for
// the stage-d frontier and build its head input in LDS.  Returns false if
// the round was abandoned.
template <int DT, int KMAX>
__device__ __forceinline__ bool stage_inputs(const Plan& p, const Plan& sp, int d,
                                             FrontShared& fs, int& sh_go) {
  if (d > 0) {
    if (threadIdx.x < 64) {
      const int ok = wait_frontier(p, d, fs);
      if (threadIdx.x == 0) sh_go = ok;
    }
    __syncthreads();
    if (!sh_go) return false;
  }
  frontier_call<DT>(sp, d);
  return true;
}

// The stage-0 frontier: each request's root (token 0 stands in for an invalid
// one, whose tree is emitted empty).
__device__ __forceinline__ void init_front(const Plan& p, FrontShared& fs) {
  for (int i = threadIdx.x; i < p.R * p.kk; i += blockDim.x) {
    const int root = p.root[i / p.kk];
    fs.tok[i] = root < 0 || root >= p.V ? 0 : root;
    fs.score[i] = 0.0f;
  }
}

// One streaming workgroup of the persistent round: a fixed V-slice whose W
// tiles stay on chip (RT per wave in registers, up to LTW per wave in LDS in
// fragment order, the rest re-read every stage), B stages of frontier
// selection + head stream + partial publication.
template <int DT, int NCMAX, int KMAX>
__device__ __forceinline__ void stream_block(const Plan& p, const Plan& sp, HeadShared<KMAX, kRoundWaves>& sh,
                             FrontShared& fs, char* ul, u32x4* wl, int& sh_go) {
  constexpr int WAVES = kRoundWaves;
  constexpr int RT = resident_reg_tiles(NCMAX);
  constexpr int LTW = resident_lds_tiles_per_wave(NCMAX);
  const int slice = blockIdx.x;
  const int t0 = slice * p.tiles_per_slice;
  const int t1 = min(t0 + p.tiles_per_slice, p.ntiles);
  const int nreg = min(t1 - t0, RT * WAVES);
  const int nlds = min(t1 - t0 - nreg, min(p.lds_tiles, LTW * WAVES));
  const int lds0 = t0 + nreg;     // first LDS-resident tile
  const int str0 = lds0 + nlds;   // first streamed tile
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;

  init_front(p, fs);
  {  // load the resident tiles (the lane geometry of A does not depend on rows)
    const HeadLane h0(p, 1, 0);
    u32x4 a[NCMAX];
    for (int j = wave; j < nlds; j += WAVES) {
      load_afrag<DT, NCMAX>(p, h0, lds0 + j, a);
#pragma unroll
      for (int c = 0; c < NCMAX; ++c) wl[((size_t)j * NCMAX + c) * 64 + lane] = a[c];
    }
  }
  u32x4 areg[RT][NCMAX];
  {
    const HeadLane h0(p, 1, 0);
#pragma unroll
    for (int i = 0; i < RT; ++i) load_afrag<DT, NCMAX>(p, h0, min(t0 + wave + WAVES * i, t1 - 1), areg[i]);
  }
  __syncthreads();

  for (int d = 0; d < p.B; ++d) {
    const int P = head_rows(p.mode, d, p.kk);
    const HeadLane h(p, P, 0);
    // frontier-independent loads before the wait
    uint32_t lreg[RT][4], llds[LTW][4];
#pragma unroll
    for (int i = 0; i < RT; ++i) load_lfrag<DT>(p, h, d, min(t0 + wave + WAVES * i, t1 - 1), lreg[i]);
#pragma unroll
    for (int q = 0; q < LTW; ++q)
      load_lfrag<DT>(p, h, d, min(lds0 + wave + WAVES * q, t1 - 1), llds[q]);
    TIMELINE_SLICE(d, 0);
    if (!stage_inputs<DT, KMAX>(p, sp, d, fs, sh_go)) return;
    TIMELINE_SLICE(d, 1);
    u32x4 bfrag[NCMAX];
    load_bfrag_lds<DT, NCMAX>(p, h, ul, bfrag);
    RowAcc<KMAX> r;
    r.init();
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      const int t = t0 + wave + WAVES * i;
      int tt = t;
      asm volatile("" : "+v"(tt));  // keep the key parts of a resident tile unhoisted
      if (t < lds0) tile_step<DT, NCMAX, KMAX>(p, h, areg[i], bfrag, lreg[i], tt, r);
    }
#pragma unroll
    for (int q = 0; q < LTW; ++q) {
      const int j = wave + WAVES * q;
      if (j < nlds) {
        u32x4 a[NCMAX];
#pragma unroll
        for (int c = 0; c < NCMAX; ++c) a[c] = wl[((size_t)j * NCMAX + c) * 64 + lane];
        int tt = lds0 + j;
        asm volatile("" : "+v"(tt));  // (as above)
        tile_step<DT, NCMAX, KMAX>(p, h, a, bfrag, llds[q], tt, r);
      }
    }
    for (int t = str0 + wave; t < t1; t += WAVES) {
      Tile<NCMAX> T;
      load_afrag<DT, NCMAX>(p, h, t, T.a);
      load_lfrag<DT>(p, h, d, t, T.l);
      tile_step<DT, NCMAX, KMAX>(p, h, T.a, bfrag, T.l, t, r);
    }
    TIMELINE_SLICE(d, 2);
    publish_partial<KMAX, WAVES>(p, h, d, slice, r, sh);
    TIMELINE_SLICE(d, 3);
  }
}

// stream_block for at most 8 frontier rows: tiles go through the MFMA in
// pairs whose C fragments are folded into one set of 16 columns (see
// HeadLane), so every lane's epilogue works on a live row.
template <int DT, int NCMAX, int KMAX>
__device__ void stream_block_fold(const Plan& p, const Plan& sp,
                                  HeadShared<KMAX, kRoundWaves>& sh, FrontShared& fs, char* ul,
                                  u32x4* wl, int& sh_go) {
  constexpr int WAVES = kRoundWaves;
  constexpr int RT = resident_reg_tiles(NCMAX, true);
  constexpr int LTW = resident_lds_tiles_per_wave(NCMAX);
  constexpr int RP = (RT + 1) / 2;   // register-resident pairs per wave
  constexpr int LP = (LTW + 1) / 2;  // LDS-resident pairs per wave
  const int slice = blockIdx.x;
  const int t0 = slice * p.tiles_per_slice;
  const int t1 = min(t0 + p.tiles_per_slice, p.ntiles);
  const int nreg = min(t1 - t0, RT * WAVES);
  const int nlds = min(t1 - t0 - nreg, min(p.lds_tiles, LTW * WAVES));
  const int lds0 = t0 + nreg;
  const int str0 = lds0 + nlds;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;

  init_front(p, fs);
  {
    const HeadLane h0(p, 1, 0);
    u32x4 a[NCMAX];
    for (int j = wave; j < nlds; j += WAVES) {
      load_afrag<DT, NCMAX>(p, h0, lds0 + j, a);
#pragma unroll
      for (int c = 0; c < NCMAX; ++c) wl[((size_t)j * NCMAX + c) * 64 + lane] = a[c];
    }
  }
  u32x4 areg[RT][NCMAX];
  {
    const HeadLane h0(p, 1, 0);
#pragma unroll
    for (int i = 0; i < RT; ++i) load_afrag<DT, NCMAX>(p, h0, min(t0 + wave + WAVES * i, t1 - 1), areg[i]);
  }
  __syncthreads();

  for (int d = 0; d < p.B; ++d) {
    const int P = head_rows(p.mode, d, p.kk);
    const HeadLane h(p, P, 0, true);
    // L_d of the lane's own tile of every resident pair, before the wait
    uint32_t lreg[RP][4], llds[LP][4];
#pragma unroll
    for (int q = 0; q < RP; ++q)
      load_lfrag<DT>(p, h, d, min(t0 + wave + WAVES * (2 * q + h.half), t1 - 1), lreg[q]);
#pragma unroll
    for (int q = 0; q < LP; ++q)
      load_lfrag<DT>(p, h, d, min(lds0 + wave + WAVES * (2 * q + h.half), t1 - 1), llds[q]);
    TIMELINE_SLICE(d, 0);
    if (!stage_inputs<DT, KMAX>(p, sp, d, fs, sh_go)) return;
    TIMELINE_SLICE(d, 1);
    u32x4 bfrag[NCMAX];
    load_bfrag_lds<DT, NCMAX>(p, h, ul, bfrag);
    RowAcc<KMAX> r;
    r.init();
#pragma unroll
    for (int q = 0; q < RP; ++q) {
      const int i1 = min(2 * q + 1, RT - 1);
      const int ta = t0 + wave + WAVES * (2 * q);
      const int tb = t0 + wave + WAVES * (2 * q + 1);
      const bool okb = 2 * q + 1 < RT && tb < lds0;
      // the tile index is the same every stage; hidden from the compiler so
      // that the token parts of its keys are recomputed (a few VALU ops)
      // rather than hoisted out of the stage loop and spilled to scratch
      int tt = h.half ? tb : ta;
      asm volatile("" : "+v"(tt));
      if (ta < lds0)
        tile_pair_step<DT, NCMAX, KMAX>(p, h, areg[2 * q], areg[i1], bfrag, lreg[q], tt,
                                        h.half ? okb : true, r);
    }
#pragma unroll
    for (int q = 0; q < LP; ++q) {
      const int ja = wave + WAVES * (2 * q);
      const int jb = wave + WAVES * (2 * q + 1);
      if (ja < nlds) {
        const bool okb = 2 * q + 1 < LTW && jb < nlds;
        const int jl = okb ? jb : ja;
        int tt = lds0 + (h.half ? jb : ja);
        asm volatile("" : "+v"(tt));  // (as above)
        lds_pair_step<DT, NCMAX, KMAX>(p, h, wl + (size_t)ja * NCMAX * 64 + lane,
                                       wl + (size_t)jl * NCMAX * 64 + lane, bfrag, llds[q], tt,
                                       h.half ? okb : true, r);
      }
    }
    for (int ta = str0 + wave; ta < t1; ta += 2 * WAVES) {
      const int tb = ta + WAVES;
      const bool okb = tb < t1;
      const int tl = h.half && okb ? tb : ta;
      u32x4 a0[NCMAX], a1[NCMAX];
      uint32_t l[4];
      load_afrag<DT, NCMAX>(p, h, ta, a0);
      load_afrag<DT, NCMAX>(p, h, okb ? tb : ta, a1);
      load_lfrag<DT>(p, h, d, tl, l);
      tile_pair_step<DT, NCMAX, KMAX>(p, h, a0, a1, bfrag, l, tl, h.half ? okb : true, r);
    }
    TIMELINE_SLICE(d, 2);
    publish_partial<KMAX, WAVES, true>(p, h, d, slice, r, sh);
    TIMELINE_SLICE(d, 3);
  }
}

// ---------------------------------------------------------------------------
// stage selection on merged rows (shared by both launch forms)
// ---------------------------------------------------------------------------
// A workgroup barrier for LDS traffic only: unlike __syncthreads() it does
// not wait for the wave's outstanding global stores.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Number of keys[0..n) greater than `key`; the loads of up to 32 entries are
// issued before any comparison (a dependent LDS read per entry, or per small
// batch, would cost its full latency over and over).
__device__ __forceinline__ int count_greater(const uint64_t* keys, int n, uint64_t key) {
  int cnt = 0;
  int c = 0;
  for (; c + 32 <= n; c += 32) {
    uint64_t v[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) v[i] = keys[c + i];
#pragma unroll
    for (int i = 0; i < 32; ++i) cnt += v[i] > key;
  }
  for (; c + 8 <= n; c += 8) {
    uint64_t v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = keys[c + i];
#pragma unroll
    for (int i = 0; i < 8; ++i) cnt += v[i] > key;
  }
  for (; c < n; ++c) cnt += keys[c] > key;
  return cnt;
}

// The number of keys[0..n) greater than `key` when keys are sorted in
// descending order: a binary search, log2(n) dependent reads instead of n.
__device__ __forceinline__ int count_greater_desc(const uint64_t* keys, int n, uint64_t key) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (keys[mid] > key)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// The same count by a group of T adjacent lanes (T a power of two <= 64):
// lane q of the group counts keys q, q + T, q + 2T, ... (the group reads T
// consecutive keys per load, no bank conflicts), eight loads in flight at a
// time, and the group adds its counts over lane swaps.  Every lane of the
// wave must call it (n = 0 for lanes without a key); each lane gets the
// group's count.
__device__ __forceinline__ int count_greater_group(const uint64_t* keys, int n, uint64_t key,
                                                   int q, int T) {
  int cnt = 0;
  for (int b = q; b < n; b += 8 * T) {
    uint64_t v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = keys[min(b + i * T, n - 1)];
#pragma unroll
    for (int i = 0; i < 8; ++i) cnt += (b + i * T < n) & (v[i] > key);
  }
  for (int m = 1; m < T; m <<= 1) cnt += __shfl_xor(cnt, m);
  return cnt;
}

// Lanes per key for count_greater_group: the largest power of two <= 64
// with n keys * T <= nthreads.
__device__ __forceinline__ int group_lanes(int n, int nthreads) {
  int T = 1;
  while (T < 64 && n * T * 2 <= nthreads) T *= 2;
  return T;
}

struct SelShared {
  int next_tok[kNarrowRows];  // tokens of the next frontier, by slot (request-major)
  uint64_t rowkeys[kNarrowRows][16];  // top-k' children (child keys) of each row
  float lse[kNarrowRows];
  __attribute__((aligned(16))) uint64_t ckey[256];  // node keys of the stage's candidates
  int rank[256];
  __attribute__((aligned(16))) uint64_t tkey[PCTREE_EMIT_MAX_N];  // a request's top-N keys
  __attribute__((aligned(16))) uint64_t sk[256];  // the surviving candidates' keys, by request
  int sci[256];         // and their candidate indices
  int rstart[17];       // each request's first survivor (and the total after the last)
  uint32_t tord[16];    // each request's survival threshold (high word of a key)
  int wcnt[kSelectThreads / 64];  // survivors per wave
  int abort;  // a wait of the selection timed out
};

// Candidates of the P rows of each request in [req0, req0 + nreq), whose
// top-k' children and lse are in sh.rowkeys / sh.lse (request-major, row 0 =
// request req0's slot 0): score them (Eq. 4), put them into the pool, pick the
// next frontier (the k' best of each request's layer, Sec. 4.1), merge them
// into the running global top-N (Sec. 4.2) and write the next head input.
// Needs blockDim >= 512 and nreq * P * k' <= 256.  `mid` runs (all threads)
// once the next frontier is in sh.next_tok and the pool entries are stored,
// before the top-N merge: a caller issues the next stage's loads there.
struct NoMid {
  __device__ void operator()() const {}
};
template <class Mid = NoMid>
__device__ __forceinline__ void stage_select_body(const Plan& p, const State& st, int d, int P,
                                                  int req0, int nreq, SelShared& sh,
                                                  bool bcast, bool shared, Mid mid = Mid()) {
  const int tid = threadIdx.x;
  const int kk = p.kk;
  const int per_req = P * kk;
  const int ncand = nreq * per_req;
  const int nbase = d == 0 ? 1 : 1 + kk + (d - 1) * kk * kk;  // pool id of the first candidate
  const bool more = d + 1 < p.B;

  int tok = 0, par = 0;
  float score = 0.0f;
  if (tid < ncand) {
    const int rq = tid / per_req;
    const int ci = tid - rq * per_req;
    const int pr = ci / kk;
    const int j = ci - pr * kk;
    const int req = req0 + rq;
    const int lrow = shared ? rq : rq * P + pr;  // shared: one row serves every parent
    const uint64_t ck = sh.rowkeys[lrow][j];
    // every row holds >= k' real keys (V >= k'); the clamp only keeps a
    // corrupted key from indexing out of bounds
    tok = min(max(child_key_token(ck), 0), p.V - 1);
    const float lp = child_key_value(ck) - sh.lse[lrow];
    score = st.front_score[(req - st.rbase) * kk + pr] + lp;
    par = st.front_node[(req - st.rbase) * kk + pr];
    sh.ckey[tid] = node_key(score, d + 1, tok, pr);
  }
  // (the frontier's loads above have returned: LDS barriers suffice until
  // the frontier is rewritten)
  lds_barrier();
  // With many candidates per request (config-sized layers of 128 and up),
  // only those that can still enter the next frontier or the running top-N
  // are ranked.  A parent's children are sorted, so its first child scores
  // highest; with P >= k' parents, the k' best candidates all score at
  // least the lowest of those P firsts.  A candidate entering a full top-N
  // scores at least its last entry.  Candidates scoring below both
  // thresholds (compared on the key's high word, the ordered score) are
  // dropped; every survivor's rank among all candidates equals its rank
  // among the survivors, and every dropped one ranks below every survivor
  // and every top-N entry.  Smaller layers are ranked whole, one thread per
  // candidate (the pruning's extra barriers cost more than they save).
  const int ncur = min(p.N, nbase);
  const bool prune = per_req >= 128;
  if (prune) {
    if (tid < nreq) {
      uint32_t tf = more ? 0u : 0xFFFFFFFFu;
      if (more && P >= kk) {
        tf = 0xFFFFFFFFu;
        for (int pr = 0; pr < P; ++pr)
          tf = min(tf, (uint32_t)(sh.ckey[tid * per_req + pr * kk] >> 32));
      }
      const uint32_t tn =
          ncur == p.N
              ? (uint32_t)(st.top_key[(size_t)(req0 + tid - st.rbase) * p.N + p.N - 1] >> 32)
              : 0u;
      sh.tord[tid] = min(tf, tn);
    }
    lds_barrier();
    // the survivors, compacted in candidate order (so each request's are
    // contiguous): wave counts, then each lane's exclusive prefix
    const int lane = tid & 63, wave = tid >> 6;
    const bool surv = tid < ncand && (uint32_t)(sh.ckey[tid] >> 32) >= sh.tord[tid / per_req];
    const uint64_t bal = __ballot(surv);
    if (lane == 0) sh.wcnt[wave] = __popcll(bal);
    lds_barrier();
    int total = 0, base = 0;
    for (int w = 0; w < (ncand + 63) / 64; ++w) {
      const int c = sh.wcnt[w];
      base += w < wave ? c : 0;
      total += c;
    }
    if (tid < ncand) {
      const int pos = base + __popcll(bal & ((1ull << lane) - 1));
      if (surv) {
        sh.sk[pos] = sh.ckey[tid];
        sh.sci[pos] = tid;
      }
      sh.rank[tid] = 0x7FFFFFFF;  // (a survivor's is set below)
      if (tid % per_req == 0) sh.rstart[tid / per_req] = pos;
    }
    if (tid == 0) sh.rstart[nreq] = total;
    lds_barrier();
    // each survivor's rank among its request's survivors, T lanes each
    const int T = group_lanes(total, blockDim.x);
    const int e = tid / T;
    const bool live = e < total;
    const int c = live ? sh.sci[e] : 0;
    const int s0 = sh.rstart[c / per_req];
    const int n = live ? sh.rstart[c / per_req + 1] - s0 : 0;
    const int cnt = count_greater_group(sh.sk + s0, n, live ? sh.sk[e] : 0, tid & (T - 1), T);
    if (live && (tid & (T - 1)) == 0) sh.rank[c] = cnt;
  } else if (tid < ncand) {
    const int rq = tid / per_req;
    sh.rank[tid] = count_greater(sh.ckey + rq * per_req, per_req, sh.ckey[tid]);
  }
  lds_barrier();
  // next frontier (every frontier slot was read above, before the barriers)
  if (more && tid < ncand && sh.rank[tid] < kk) {
    const int rq = tid / per_req;
    const int ci = tid - rq * per_req;
    const int req = req0 + rq;
    const int slot = sh.rank[tid];
    if (bcast) {  // the streaming workgroups wait for these words
      // (with one shared row, the next row's token is the greedy chain's:
      // the row's best child, which slot 0 carries)
      const int wtok = shared ? min(max(child_key_token(sh.rowkeys[rq][0]), 0), p.V - 1) : tok;
      __hip_atomic_store(p.front_w + (size_t)(d + 1) * p.rows_max + req * kk + slot,
                         ((uint64_t)__float_as_uint(score) << 32) |
                             ((uint64_t)wtok << kTagBits) | p.tag,
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    st.front_node[(req - st.rbase) * kk + slot] = nbase + ci;
    st.front_tok[(req - st.rbase) * kk + slot] = tok;
    st.front_score[(req - st.rbase) * kk + slot] = score;
    if (rq * kk + slot < kNarrowRows) sh.next_tok[rq * kk + slot] = tok;
    if (p.t_token) {
      const size_t o = ((size_t)req * p.B + d + 1) * p.k + slot;
      p.t_token[o] = tok;
      p.t_pslot[o] = ci / kk;
      p.t_score[o] = score;
    }
  }
  // the pool entries of the stage's candidates
  if (tid < ncand) {
    const int rq = tid / per_req;
    const size_t id = (size_t)(req0 + rq) * p.maxpool + nbase + (tid - rq * per_req);
    p.node_tok[id] = tok;
    p.node_par[id] = par;
    p.node_depth[id] = d + 1;
    p.node_score[id] = score;
  }
  mid();
  // running global top-N, one request at a time: every element's new
  // position is its rank in the union (both sides are sorted), computed
  // before any element moves.  The state is in LDS (every caller keeps a
  // copy there), so LDS barriers order it; the global stores above need no
  // wait until the barrier that ends the stage.
  for (int rq = 0; rq < nreq; ++rq) {
    const int req = req0 + rq;
    uint64_t* tk = st.top_key + (size_t)(req - st.rbase) * p.N;
    int* tn = st.top_node + (size_t)(req - st.rbase) * p.N;
    lds_barrier();
    for (int i = tid; i < ncur; i += blockDim.x) sh.tkey[i] = tk[i];
    lds_barrier();
    // the request's candidates: its survivors, or all of them
    const int s0 = prune ? sh.rstart[rq] : rq * per_req;
    const int ns = prune ? sh.rstart[rq + 1] - s0 : per_req;
    const uint64_t* keys = prune ? sh.sk : sh.ckey;
    int pos = p.N, node = 0;
    uint64_t key = 0;
    if (tid < ns) {
      const int c = prune ? sh.sci[s0 + tid] : s0 + tid;
      key = keys[s0 + tid];
      pos = sh.rank[c] + count_greater_desc(sh.tkey, ncur, key);  // (the top-N is sorted)
      node = nbase + c - rq * per_req;
    } else if (tid >= 256 && tid < 256 + ncur) {
      const int i = tid - 256;
      key = sh.tkey[i];
      pos = i + count_greater(keys + s0, ns, key);
      node = tn[i];
    }
    lds_barrier();
    if (pos < p.N) {
      tk[pos] = key;
      tn[pos] = node;
    }
  }
  // (the stage's global stores, pool entries and trace, are read by later
  // launches or, in the persistent form, by the emission after a full
  // barrier: an LDS barrier ends the stage)
  lds_barrier();
}

// The stage, init and emission routines have an out-of-line entry (used by the
// multi-launch kernels and the k' <= 8 keepers) and an inlined body: a keeper
// with k' = 16 that called them out of line kept a copy of its launch
// arguments in scratch memory, so it inlines the bodies instead.
__device__ void stage_select(const Plan& p, const State& st, int d, int P, int req0, int nreq,
                             SelShared& sh, bool bcast, bool shared = false) {
  stage_select_body(p, st, d, P, req0, nreq, sh, bcast, shared);
}

// The top-k' children and the lse of each of the R*P (<= 16) rows of stage d
// from the published slice partials, one wave per row, as the words land:
// every word carries the call's tag, so the wave re-reads (agent-coherent
// loads) the records that are not complete yet until all are.  Every slice's
// record holds its kHeadKeys best keys and its sum of exp: k' pops of the
// wave-wide maximum over the union of those keys give the row's top-k' unless
// some slice gave up all of its record keys (it may hold more that belong).
// Then, and only then, the lists are read: a row's top-k' lie in the k'
// slices with the largest best keys (any other slice is beaten k' times
// over), and k' pops over those lists give the exact answer.  Keys are unique
// (the token is part of them), so each pop removes exactly one entry.
// Returns false if a wait ran past p.spin_ticks (the round is abandoned).
template <int KMAX, int HPL>
__device__ __forceinline__ bool sel_merge_rows(const Plan& p, int d, int rows, SelShared& sh) {
  constexpr int HK = KMAX < kHeadKeys ? KMAX : kHeadKeys;  // record keys that can be real
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwave = blockDim.x >> 6;
  const int G = p.G;
  const int kk = p.kk;
  bool alive = true;
  for (int row = wave; row < rows && alive; row += nwave) {
    const size_t base = ((size_t)d * p.rows_max + row) * kSlicesMax;
    const uint64_t* recs = slice_record(p, d, row);
    uint64_t hk[HPL][HK], first[HPL];
    float hs[HPL];
    bool have[HPL];
#pragma unroll
    for (int c = 0; c < HPL; ++c) {
      have[c] = lane + 64 * c >= G;  // no slice: nothing to wait for
#pragma unroll
      for (int i = 0; i < HK; ++i) hk[c][i] = 0;
      hs[c] = 0.0f;
    }
    const long long t0 = wall_clock64();
    for (;;) {
#pragma unroll
      for (int c = 0; c < HPL; ++c) {
        if (!have[c]) {
          const uint64_t* rec = recs + lane + 64 * c;
          uint64_t w[kRecWords];
#pragma unroll
          for (int i = 0; i < kRecWords; ++i) w[i] = load_agent(rec + i * kSlicesMax);
          bool ok = sum_tagged(p, w[kHeadKeys]);
#pragma unroll
          for (int i = 0; i < kHeadKeys; ++i) ok = ok && key_tagged(p, w[i]);
          have[c] = ok;
#pragma unroll
          for (int i = 0; i < HK; ++i) hk[c][i] = w[i];
          hs[c] = __uint_as_float((uint32_t)w[kHeadKeys]);
        }
      }
      bool all = true;
#pragma unroll
      for (int c = 0; c < HPL; ++c) all = all && have[c];
      if (__all(all)) break;
      if (wall_clock64() - t0 > p.spin_ticks) {
        alive = false;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (!alive) break;
    // lse over the slices: each sum is relative to the slice's best logit
    float m = kNegBig, s = 0.0f;
#pragma unroll
    for (int c = 0; c < HPL; ++c) {
      first[c] = hk[c][0];
      if (lane + 64 * c < G) lse_combine(m, s, child_key_value(hk[c][0]), hs[c]);
    }
    const float M = wave_max_f32(m);
    const float S = wave_sum_f32(s * exp2_raw((m - M) * kLog2e));
    int used[HPL];
#pragma unroll
    for (int c = 0; c < HPL; ++c) used[c] = 0;
#pragma unroll
    for (int it = 0; it < KMAX; ++it) {
      if (it < kk) {
        uint64_t lm = hk[0][0];
#pragma unroll
        for (int c = 1; c < HPL; ++c) lm = key_max(lm, hk[c][0]);
        const uint64_t best = wave_max_u64(lm);
#pragma unroll
        for (int c = 0; c < HPL; ++c) {
          if (hk[c][0] == best) {
#pragma unroll
            for (int i = 0; i + 1 < HK; ++i) hk[c][i] = hk[c][i + 1];
            hk[c][HK - 1] = 0;
            ++used[c];
          }
        }
        if (lane == 0) sh.rowkeys[row][it] = best;
      }
    }
    // (pops past the union's real keys return 0 and count for every empty
    // entry, so a slice's count can pass HK)
    bool gave_all = false;
    if (HK < KMAX) {
#pragma unroll
      for (int c = 0; c < HPL; ++c) gave_all = gave_all || used[c] >= HK;
    }
    if (__any(gave_all)) {
      // the k' largest best keys; lane i keeps the slice of the i-th
      const int nwin = min(kk, G);
#pragma unroll
      for (int c = 1; c < HPL; ++c) {
#pragma unroll
        for (int i = c; i > 0; --i) {
          const uint64_t a = first[i - 1], b = first[i];
          const bool sw = b > a;
          first[i - 1] = sw ? b : a;
          first[i] = sw ? a : b;
        }
      }
      uint64_t won = 0;
#pragma unroll
      for (int it = 0; it < KMAX; ++it) {
        if (it < nwin) {
          const uint64_t best = wave_max_u64(first[0]);
          if (first[0] == best) {
#pragma unroll
            for (int c = 0; c + 1 < HPL; ++c) first[c] = first[c + 1];
            first[HPL - 1] = 0;
          }
          if (lane == it) won = best;
        }
      }
      const int myslice =
          lane < nwin ? min(child_key_token(won) / (p.tiles_per_slice * kTile), G - 1) : 0;
      const uint64_t* src = p.part_key + (base + myslice) * KMAX;
      uint64_t lst[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) lst[i] = 0;
      bool got = lane >= nwin;
      const long long t1 = wall_clock64();
      for (;;) {
        if (!got) {
          bool ok = true;
#pragma unroll
          for (int i = 0; i < KMAX; ++i) {
            lst[i] = load_agent(src + i);
            ok = ok && key_tagged(p, lst[i]);
          }
          got = ok;
        }
        if (__all(got)) break;
        if (wall_clock64() - t1 > p.spin_ticks) {
          alive = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      if (!alive) break;
      if (lane >= nwin) {
#pragma unroll
        for (int i = 0; i < KMAX; ++i) lst[i] = 0;
      }
#pragma unroll
      for (int it = 0; it < KMAX; ++it) {
        if (it < kk) {
          const uint64_t best = wave_max_u64(lst[0]);
          if (lst[0] == best) {
#pragma unroll
            for (int i = 0; i + 1 < KMAX; ++i) lst[i] = lst[i + 1];
            lst[KMAX - 1] = 0;
          }
          if (lane == 0) sh.rowkeys[row][it] = best;
        }
      }
    }
    if (lane == 0) sh.lse[row] = M + logf(S);
  }
  if (!alive && lane == 0) sh.abort = 1;
  __syncthreads();
  return sh.abort == 0;
}

// The persistent form uses at most kRoundSlicesMax slices (one per CU).
template <int KMAX>
__device__ __forceinline__ bool sel_merge(const Plan& p, int d, int rows, SelShared& sh) {
  if (p.G <= 64) return sel_merge_rows<KMAX, 1>(p, d, rows, sh);
  if (p.G <= 128) return sel_merge_rows<KMAX, 2>(p, d, rows, sh);
  return sel_merge_rows<KMAX, kRoundSlicesMax / 64>(p, d, rows, sh);
}


// ---------------------------------------------------------------------------
// emission in canonical order (+ optional ancestor mask)
// ---------------------------------------------------------------------------
// Row i of the ancestor mask = i and its ancestors (App. A).  One row per
// thread at a time, built in `scratch` (stride words per thread).
__device__ void mask_rows(const int* par, int count, int N, uint32_t* out, uint32_t* scratch,
                          int stride) {
  const int nw = (N + 31) / 32;
  uint32_t* w = scratch + threadIdx.x * stride;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    for (int q = 0; q < nw; ++q) w[q] = 0u;
    if (i < count) {
      int j = i;
      while (j >= 0) {
        w[j >> 5] |= 1u << (j & 31);
        const int pj = par[j];
        if (pj >= j || pj < -1) break;  // not a valid parent index: end the walk
        j = pj;
      }
    }
    for (int q = 0; q < nw; ++q) out[(size_t)i * nw + q] = w[q];
  }
}

// Canonical order: depth ascending, then (parent's emitted index, token).
// Level by level, every node of the level ranks itself among its level by
// the key (emitted index of its parent + 1) << 20 | token, written to a
// dense slot of the level (tokens < 2^20, indices < 2^11).  Each node finds
// its parent among the selected nodes of the level above once, up front.
// The global reads (the request's flags and the selected nodes' pool
// entries) are issued together, and the LDS loops issue their reads in
// batches of 8 (a dependent LDS read per step would cost its full latency
// every time).  The ancestor mask row of a node is its parent's row (done a
// level earlier) plus its own bit.  Uses threads [0, 256) of the block
// (N <= 256); all threads must call it.
__device__ __forceinline__ void emit_request_body(const Plan& p, const State& st, int req) {
  constexpr int kBatch = 8;
  __shared__ int sh_node[kEmitThreads], sh_emit[kEmitThreads];
  __shared__ int sh_td[kEmitThreads];     // depth << 20 | token
  __shared__ uint32_t sh_lkey[kEmitThreads];  // level keys, by level slot
  __shared__ int lev_cnt[64], lev_off[65], lev_fill[64];
  __shared__ int sh_maxdep;
  __shared__ uint32_t sh_words[kEmitThreads * (PCTREE_EMIT_MAX_N / 32)];  // mask rows

  const int tid = threadIdx.x;
  const int kk = p.kk;
  const int pool = 1 + kk + (p.B - 1) * kk * kk;
  const int count0 = min(p.N, pool);
  const size_t pb = (size_t)req * p.maxpool;

  // every global read at once: the request's flags and the pool entries of
  // the first count0 selected nodes (the top-N ids live in LDS)
  const int bad = p.req_bad[req];
  const int prefix = p.prefix[req];
  int node = -1, dep = -1, tok = -1, pnode = -1;
  float score = 0.0f;
  if (tid < count0) {
    // (clamped: an inconsistent state must not address outside the pool)
    node = min(max(st.top_node[(size_t)(req - st.rbase) * p.N + tid], 0), p.maxpool - 1);
    dep = p.node_depth[pb + node];
    tok = p.node_tok[pb + node];
    pnode = p.node_par[pb + node];
    score = p.node_score[pb + node];
  }
  const int count = bad ? 0 : count0;

  __syncthreads();
  if (tid < 64) {
    lev_cnt[tid] = 0;
    lev_fill[tid] = 0;
  }
  if (tid == 0) sh_maxdep = -1;
  __syncthreads();
  const bool mine = tid < count;
  if (mine) {
    dep = min(max(dep, 0), p.B);
    sh_node[tid] = node;
    sh_td[tid] = (dep << 20) | (tok & 0xFFFFF);
    atomicAdd(&lev_cnt[dep], 1);
    atomicMax(&sh_maxdep, dep);
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int l = 0; l <= p.B; ++l) {
      lev_off[l] = acc;
      acc += lev_cnt[l];
    }
    lev_off[p.B + 1] = acc;
  }
  // the parent among the selected nodes one level up (-1: none)
  int pidx = -1;
  if (mine && dep > 0) {
    const int want = (dep - 1) << 20;
    for (int j0 = 0; j0 < count; j0 += kBatch) {
      int nd[kBatch], td[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int j = min(j0 + i, count - 1);
        nd[i] = sh_node[j];
        td[i] = sh_td[j];
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i)
        if (j0 + i < count && nd[i] == pnode && (td[i] & ~0xFFFFF) == want) pidx = j0 + i;
    }
  }
  __syncthreads();  // lev_off
  const int myslot = mine ? lev_off[dep] + atomicAdd(&lev_fill[dep], 1) : -1;

  int emit = -1, pemit = -1;
  const int maxdep = sh_maxdep;
  constexpr int MW = PCTREE_EMIT_MAX_N / 32;  // mask words of a row in LDS
  const int nw = (p.N + 31) / 32;
  for (int l = 0; l <= maxdep; ++l) {
    const bool here = mine && dep == l;
    uint32_t key = 0;
    if (here) {
      pemit = pidx >= 0 ? sh_emit[pidx] : -1;
      key = ((uint32_t)(pemit + 1) << 20) | (uint32_t)(tok & 0xFFFFF);
      sh_lkey[myslot] = key;
    }
    __syncthreads();
    if (here) {
      const int q0 = lev_off[l], q1 = lev_off[l + 1];
      int rank = 0;
      for (int q = q0; q < q1; q += kBatch) {
        uint32_t k8[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) k8[i] = sh_lkey[min(q + i, q1 - 1)];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) rank += (q + i < q1) && k8[i] < key;
      }
      emit = q0 + rank;
      sh_emit[tid] = emit;
      if (p.o_mask) {
        for (int w = 0; w < nw; ++w) {
          const uint32_t up = pemit >= 0 ? sh_words[pemit * MW + w] : 0u;
          sh_words[emit * MW + w] = up | (w == (emit >> 5) ? 1u << (emit & 31) : 0u);
        }
      }
    }
    __syncthreads();
  }

  const size_t ob = (size_t)req * p.N;
  if (mine) {
    p.o_token[ob + emit] = tok;
    p.o_parent[ob + emit] = pemit;
    p.o_depth[ob + emit] = dep;
    p.o_position[ob + emit] = prefix + dep;
    p.o_logprob[ob + emit] = score;
  }
  for (int e = count + tid; e < p.N; e += blockDim.x) {
    p.o_token[ob + e] = -1;
    p.o_parent[ob + e] = -1;
    p.o_depth[ob + e] = -1;
    p.o_position[ob + e] = -1;
    p.o_logprob[ob + e] = -INFINITY;
  }
  if (tid == 0) p.o_count[req] = count;
  if (p.o_mask) {
    uint32_t* out = p.o_mask + (size_t)req * p.N * nw;
    for (int e = tid; e < p.N; e += blockDim.x)
      for (int w = 0; w < nw; ++w) out[(size_t)e * nw + w] = e < count ? sh_words[e * MW + w] : 0u;
  }
  __syncthreads();
}

__device__ void emit_request(const Plan& p, const State& st, int req) {
  emit_request_body(p, st, req);
}

// An abandoned round (a bounded wait ran out): every output row of every
// request is written as padding, mask rows zero, and count = -1 marks the
// abort, so that nothing of an earlier call's tree is left behind.  All
// threads of the workgroup take part.
__device__ __forceinline__ void abort_outputs(const Plan& p) {
  const int n = p.R * p.N;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    p.o_token[e] = -1;
    p.o_parent[e] = -1;
    p.o_depth[e] = -1;
    p.o_position[e] = -1;
    p.o_logprob[e] = -INFINITY;
  }
  if (p.o_mask) {
    const size_t nw = (size_t)n * ((p.N + 31) / 32);
    for (size_t e = threadIdx.x; e < nw; e += blockDim.x) p.o_mask[e] = 0u;
  }
  for (int req = threadIdx.x; req < p.R; req += blockDim.x) p.o_count[req] = -1;
}

// LDS of the persistent round kernel shared by its stage code.
__shared__ SelShared g_sel;
__shared__ FrontShared g_front;
// dynamic LDS: the frontier's head input (streaming blocks), the keeper's
// running top-N, the streaming blocks' resident W tiles
extern __shared__ uint64_t g_dyn[];

// The plan in scalar registers (read from its LDS copy): uniform loop bounds
// and addresses in the out-of-line stage code below.
__device__ __forceinline__ Plan scalar_plan(const Plan& lp) {
  static_assert(sizeof(Plan) % 4 == 0, "Plan is copied word by word");
  Plan p;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(Plan) / 4); ++i)
    ((int*)&p)[i] = __builtin_amdgcn_readfirstlane(((const int*)&lp)[i]);
  return p;
}

// The head-input code runs out of line with the plan read from an LDS copy:
// its registers do not count against the W tiles the streaming loop keeps
// resident.  The LDS objects are named directly (not passed), so that
// accesses stay LDS ones.
template <int DT>
__device__ __noinline__ void frontier_call(const Plan& lp, int d) {
  const Plan p = scalar_plan(lp);
  compute_u<DT>(p, g_front, d, head_rows(p.mode, d, p.kk), (char*)g_dyn);
}

// Blocks [0, G) stream one V-slice each; block G is the keeper.  A streaming
// block publishes the stage-d partial of its slice as tagged words (no
// ordering, no flag) and, for stage d+1, waits for the frontier words that
// the keeper publishes.  The keeper waits for all slice partials of stage d
// (re-reading the records that are not complete yet), merges them, selects
// the stage-(d+1) frontier and publishes it first; then it keeps the pool,
// the trace and the running top-N (in LDS), and emits the tree after the last
// stage.  All cross-workgroup words are written and read with agent-coherent
// (L2-bypassing) accesses; each word is valid on its own, so no fence is
// needed anywhere.  The tagged buffers are cleared before every call.
template <int DT, int NCMAX, int KMAX, bool FOLD>
__global__ __launch_bounds__(kRoundWaves * 64) void round_kernel(Plan p) {
  __shared__ int sh_go;
  SelShared& ssh = g_sel;
  char* dyn = (char*)g_dyn;
  if (blockIdx.x < p.G) {
    __shared__ HeadShared<KMAX, kRoundWaves> hsh;
    FrontShared& fs = g_front;
    __shared__ Plan sp;  // read by the out-of-line stage code
    if (threadIdx.x == 0) sp = p;
    u32x4* wl = (u32x4*)(dyn + p.lds_tile_offset);
    if constexpr (FOLD)
      stream_block_fold<DT, NCMAX, KMAX>(p, sp, hsh, fs, dyn, wl, sh_go);
    else
      stream_block<DT, NCMAX, KMAX>(p, sp, hsh, fs, dyn, wl, sh_go);
    return;
  }

  // the keeper
  __shared__ int s_front_node[kNarrowRows], s_front_tok[kNarrowRows];
  __shared__ float s_front_score[kNarrowRows];
  uint64_t* s_top = (uint64_t*)(dyn + p.lds_top_offset);
  const State st{s_front_node, s_front_tok, s_front_score, s_top,
                 (int*)(s_top + (size_t)p.R * p.N), 0};
  constexpr bool kInline = KMAX > 8;  // keeps the launch arguments out of scratch
  for (int req = 0; req < p.R; ++req) {
    if constexpr (kInline)
      init_request_body(p, req, threadIdx.x, blockDim.x);
    else
      init_request(p, req, threadIdx.x, blockDim.x);
  }
  for (int i = threadIdx.x; i < p.R * p.kk; i += blockDim.x) {
    const int r0 = p.root[i / p.kk];
    st.front_node[i] = 0;
    st.front_tok[i] = r0 < 0 || r0 >= p.V ? 0 : r0;
    st.front_score[i] = 0.0f;
  }
  for (int req = threadIdx.x; req < p.R; req += blockDim.x) {
    const int r0 = p.root[req];
    const int root = r0 < 0 || r0 >= p.V ? 0 : r0;
    st.top_key[(size_t)req * p.N] = node_key(0.0f, 0, root, 0);
    st.top_node[(size_t)req * p.N] = 0;
  }
  if (threadIdx.x == 0) ssh.abort = 0;
  __syncthreads();
  for (int d = 0; d < p.B; ++d) {
    // head rows of the stage (one per request in the control modes) and
    // frontier parents (Sec. 5.3: the control modes' one row serves them all)
    const int Ph = head_rows(p.mode, d, p.kk), Pf = d == 0 ? 1 : p.kk;
    TIMELINE_STAMP(0, d, 0);
    if (!sel_merge<KMAX>(p, d, p.R * Ph, ssh)) {
      abort_outputs(p);
      return;
    }
    TIMELINE_STAMP(0, d, 1);
    if constexpr (kInline)
      stage_select_body(p, st, d, Pf, 0, p.R, ssh, true, p.mode != 0);
    else
      stage_select(p, st, d, Pf, 0, p.R, ssh, true, p.mode != 0);
    TIMELINE_STAMP(0, d, 2);
  }
  __syncthreads();  // the pool entries stored by the stages are visible to every wave
  TIMELINE_STAMP(0, kTimelineStages - 1, 0);
  for (int req = 0; req < p.R; ++req) {
    if constexpr (kInline)
      emit_request_body(p, st, req);
    else
      emit_request(p, st, req);
  }
  TIMELINE_STAMP(0, kTimelineStages - 1, 1);
}

// ---------------------------------------------------------------------------
// wide form: per-stage head and select launches
// ---------------------------------------------------------------------------
template <int DT, int NCMAX, int KMAX>
__global__ __launch_bounds__(kHeadThreads) void head_kernel(Plan p, int d, int P) {
  __shared__ HeadShared<KMAX, kHeadThreads / 64> hsh;
  // Workgroups go to the 8 XCDs in turn (id i to XCD i % 8).  The column
  // blocks of one V-slice get consecutive ids within one XCD, so they run
  // side by side there and all but the first read the slice's W from that
  // XCD's L2.  The grid has 8 * ceil(G / 8) * ncb workgroups.
  const int ncb = (p.R * P + kTile - 1) / kTile;
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int cb = j % ncb;
  const int slice = (j / ncb) * 8 + x;
  if (slice >= p.G) return;
  head_slice<DT, NCMAX, KMAX, kHeadThreads / 64>(p, d, P, cb, slice, hsh);
}

// ---------------------------------------------------------------------------
// wide stages (more than 16 frontier rows): per-row bounds from probe tokens
// ---------------------------------------------------------------------------
// A row's k' children are its k' best logits.  Any k' logits of the row are
// at most as large as the k'-th best, so the k'-th best of the row's logits
// at a few probe tokens is a lower bound tau of it: a token whose logit lies
// below tau cannot be a child.  The probe tokens of a (request, depth) are
// about the kProbe largest base logits L_d (found once per round); the head
// stream of a wide stage then keeps, per row, the online (max, sum of exp)
// of every logit but only the rare logits at or above tau.  The bound is
// lowered by a margin that covers the difference between the probe's
// float32 dot products and the MFMA's (both sum r bf16 products in float32,
// in different orders).

// Probe tokens of every (request, depth): each thread keeps the largest base
// logit among the tokens it scans (ties: lowest id), each wave the kProbeWave
// best of its threads', and the kProbe best of those become the probes
// (fewer when V < kProbe).  Any tokens would give a valid bound; these make
// it tight.
constexpr int kProbeThreads = 1024;
constexpr int kProbeWave = 4;

__device__ __forceinline__ uint64_t probe_key(float z, int v) {
  return ((uint64_t)f32_ord(z) << 32) | (uint32_t)(0x7FFFFFFF - v);
}

template <int DT>
__device__ __forceinline__ uint64_t probe_scan(const Plan& p, size_t base) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int PER = 16 / ES;  // elements per 16-byte load
  const int tid = threadIdx.x;
  uint64_t k = 0;
  // elements before the first 16-byte boundary of the row, and after the last
  const int head = (int)(((16 - (base * ES) % 16) % 16) / ES);
  const int nvec = (p.V - min(head, p.V)) / PER;
  const int tail0 = head + nvec * PER;
  if (tid < head && tid < p.V) k = probe_key(load_elem<DT>(p.L, base + tid), tid);
  if (tail0 + tid < p.V) {
    const int v = tail0 + tid;
    const uint64_t c = probe_key(load_elem<DT>(p.L, base + v), v);
    k = c > k ? c : k;
  }
  // the aligned body: the thread's best logit and its token, compared as
  // floats in increasing token order (a strict comparison keeps the lowest
  // token of equal logits, as the key order does; -0 equals +0 in both)
  const u32x4* vec = (const u32x4*)((const char*)p.L + (base + head) * ES);
  constexpr int kBatch = 8;  // loads issued before any is used
  float bz = -INFINITY;
  int bv = -1;
  for (int c0 = 0; c0 < nvec; c0 += kBatch * kProbeThreads) {
    u32x4 w[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) w[b] = vec[min(c0 + b * kProbeThreads + tid, max(nvec - 1, 0))];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int c = c0 + b * kProbeThreads + tid;
      if (c < nvec) {
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const uint32_t word = w[b][e * ES / 4];
          const float z = DT ? __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16))
                             : __uint_as_float(word);
          const bool up = z > bz || bv < 0;
          bz = up ? z : bz;
          bv = up ? head + c * PER + e : bv;
        }
      }
    }
  }
  if (bv >= 0) {
    const uint64_t key = probe_key(bz, bv);
    k = key > k ? key : k;
  }
  return k;
}

__global__ __launch_bounds__(kProbeThreads) void probe_kernel(Plan p) {
  constexpr int NW = kProbeThreads / 64;
  __shared__ uint64_t best[NW * kProbeWave];
  const int rd = blockIdx.x;  // request * B + depth
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t k = p.dtype ? probe_scan<1>(p, (size_t)rd * p.V) : probe_scan<0>(p, (size_t)rd * p.V);
#pragma unroll
  for (int i = 0; i < kProbeWave; ++i) {
    const uint64_t m = wave_max_u64(k);
    if (k == m) k = 0;  // keys are unique: one lane gives its key up
    if (lane == 0) best[wave * kProbeWave + i] = m;
  }
  __syncthreads();
  // the kProbe best keys at their ranks; slots past the keys found (few
  // tokens reach few waves) hold -1 and are no probe
  __shared__ int toks[kProbe];
  if (threadIdx.x < NW * kProbeWave) {
    const uint64_t key = best[threadIdx.x];
    const int rank = count_greater(best, NW * kProbeWave, key);
    const int found = count_greater(best, NW * kProbeWave, 0ull);
    if (key != 0 && rank < kProbe) toks[rank] = 0x7FFFFFFF - (int)(uint32_t)key;
    if (threadIdx.x >= found && threadIdx.x < kProbe) toks[threadIdx.x] = -1;
  }
  __syncthreads();
  // their tokens, W rows (zero rows for missing probes) and base logits,
  // gathered once for the bounds of this (request, depth)
  const int words = p.r * (p.dtype ? 2 : 4) / 4;
  if (threadIdx.x < kProbe) {
    const int t = toks[threadIdx.x];
    p.probe_tok[(size_t)rd * kProbe + threadIdx.x] = t;
    p.probe_l[(size_t)rd * kProbe + threadIdx.x] =
        t < 0 ? 0.0f : (p.dtype ? load_elem<1>(p.L, (size_t)rd * p.V + t)
                                : load_elem<0>(p.L, (size_t)rd * p.V + t));
  }
  uint32_t* dst = (uint32_t*)p.probe_w + (size_t)rd * kProbe * words;
  for (int e = threadIdx.x; e < kProbe * words; e += blockDim.x) {
    const int q = e / words, j = e - q * words;
    const int t = toks[q];
    dst[e] = t < 0 ? 0u : ((const uint32_t*)p.Wt)[(size_t)t * words + j];
  }
}

// LDS of the per-request select kernels beyond the selection: the next
// stage's head input rows (32-bit words) and the probe logits.
constexpr int kProbeRowWords = 256 + 4;  // a W row of at most 1 KB, padded by 16 bytes
constexpr int kProbeSplit = 2;  // waves sharing one probe tile's chunks

struct NextShared {
  // the request's selection state: a copy of its workspace entries
  int front_node[kNarrowRows], front_tok[kNarrowRows];
  float front_score[kNarrowRows];
  __attribute__((aligned(16))) uint64_t top_key[PCTREE_EMIT_MAX_N];
  int top_node[PCTREE_EMIT_MAX_N];
  // the next stage's depth feature and probes, fetched before they are needed
  __attribute__((aligned(16))) float h[PCTREE_MAX_RANK_BF16];
  __attribute__((aligned(16))) uint32_t pw[kProbe * kProbeRowWords];
  float pl[kProbe];
  int pt[kProbe];
  // the next stage's head input rows and probe logits
  __attribute__((aligned(16))) uint32_t u[kNarrowRows * 256];  // rows of at most 1 KB
  __attribute__((aligned(16))) float zl[kNarrowRows * kProbe];
  float al[kNarrowRows * kProbe];
  // the probe logits' per-wave shares: [tile][share][token][row]
  float pz[2 * kProbeSplit * kTile * kTile], pa[2 * kProbeSplit * kTile * kTile];
};

// Loads of a request's select kernel that do not depend on the stage's
// rows, issued first so that they land while the rows merge: the request's
// selection state (frontier, running top-N) and the next stage's depth
// feature, probe tokens, probe W rows and probe base logits.  All threads
// call it; the caller synchronises before using nx.
__device__ void tail_prefetch(const Plan& p, int d, int req, NextShared& nx) {
  const int tid = threadIdx.x, nth = blockDim.x;
  const bool more = d + 1 < p.B;
  const bool probes = more && stage_wide(p.mode, d + 1, p.R, p.kk) && !p.unbounded;
  const int words = p.r * (p.dtype ? 2 : 4) / 4;
  const int units = kProbe * words / 4;  // 16-byte units of the probe rows
  const size_t pb = ((size_t)req * p.B + d + 1) * kProbe;
  const float* hrow = p.h + ((size_t)req * p.B + d + 1) * p.r;
  const u32x4* src = (const u32x4*)p.probe_w + pb * words / 4;
  // the thread's first two entries of every kind: all loads first, then the
  // LDS stores (a load and its store in turn would pay one latency per kind)
  int fn = 0, ft = 0;
  float fs = 0.0f, hv[2] = {0.0f, 0.0f}, pl = 0.0f;
  uint64_t tk[2] = {0, 0};
  int tn[2] = {0, 0}, pt = 0;
  u32x4 pw[2];
  if (tid < p.kk) {
    fn = p.front_node[req * p.kk + tid];
    ft = p.front_tok[req * p.kk + tid];
    fs = p.front_score[req * p.kk + tid];
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + k * nth;
    if (i < p.N) {
      tk[k] = p.top_key[(size_t)req * p.N + i];
      tn[k] = p.top_node[(size_t)req * p.N + i];
    }
    if (more && i < p.r) hv[k] = hrow[i];
    if (probes && i < units) pw[k] = src[i];
  }
  if (probes && tid < kProbe) {
    pt = p.probe_tok[pb + tid];
    pl = p.probe_l[pb + tid];
  }
  if (tid < p.kk) {
    nx.front_node[tid] = fn;
    nx.front_tok[tid] = ft;
    nx.front_score[tid] = fs;
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + k * nth;
    if (i < p.N) {
      nx.top_key[i] = tk[k];
      nx.top_node[i] = tn[k];
    }
    if (more && i < p.r) nx.h[i] = hv[k];
    if (probes && i < units) {
      const int q = i / (words / 4);
      *(u32x4*)&nx.pw[q * kProbeRowWords + 4 * (i - q * (words / 4))] = pw[k];
    }
  }
  if (probes && tid < kProbe) {
    nx.pt[tid] = pt;
    nx.pl[tid] = pl;
  }
  // the rest (blocks of fewer threads)
  for (int i = tid + 2 * nth; i < p.N; i += nth) {
    nx.top_key[i] = p.top_key[(size_t)req * p.N + i];
    nx.top_node[i] = p.top_node[(size_t)req * p.N + i];
  }
  if (more)
    for (int i = tid + 2 * nth; i < p.r; i += nth) nx.h[i] = hrow[i];
  if (probes)
    for (int i = tid + 2 * nth; i < units; i += nth) {
      const int q = i / (words / 4);
      *(u32x4*)&nx.pw[q * kProbeRowWords + 4 * (i - q * (words / 4))] = src[i];
    }
}

// The request's selection state back to the workspace after its stage.
__device__ void tail_writeback(const Plan& p, int req, const NextShared& nx) {
  const int tid = threadIdx.x, nth = blockDim.x;
  for (int i = tid; i < p.kk; i += nth) {
    p.front_node[req * p.kk + i] = nx.front_node[i];
    p.front_tok[req * p.kk + i] = nx.front_tok[i];
    p.front_score[req * p.kk + i] = nx.front_score[i];
  }
  for (int i = tid; i < p.N; i += nth) {
    p.top_key[(size_t)req * p.N + i] = nx.top_key[i];
    p.top_node[(size_t)req * p.N + i] = nx.top_node[i];
  }
}

// Head input of the P rows of request `req` at stage d into p.U and into
// nx.u: u = act(E[tok] + h_d) for the rows' tokens toks[0..P) (mode 2: zero
// rows).  Sixteen bytes of u per work item: their E and h loads are issued
// together.  All threads of the workgroup call it.
__device__ __forceinline__ u32x4 next_e_unit(const Plan& p, int e, const int* toks) {
  const int words = p.r * (p.dtype ? 2 : 4) / 4;
  const int s = e / (words / 4), k = e - s * (words / 4);
  const int tok = min(max(toks[s], 0), p.V - 1);
  return *(const u32x4*)((const uint32_t*)p.E + (size_t)tok * words + 4 * k);
}

// The E bytes of the thread's first unit of next_inputs, loaded ahead (zero
// when the thread has none, or in mode 2).
__device__ __forceinline__ u32x4 next_e_first(const Plan& p, int P, const int* toks) {
  const int units = P * (p.r * (p.dtype ? 2 : 4) / 16);
  return p.mode != 2 && (int)threadIdx.x < units ? next_e_unit(p, threadIdx.x, toks)
                                                 : u32x4{0u, 0u, 0u, 0u};
}

// (first: the thread's first unit's E bytes from next_e_first, or null)
__device__ void next_inputs(const Plan& p, int d, int P, int req, const int* toks, NextShared& nx,
                            const u32x4* first = nullptr) {
  const int words = p.r * (p.dtype ? 2 : 4) / 4;  // multiple of 16
  const int units = P * (words / 4);
  for (int e = threadIdx.x; e < units; e += blockDim.x) {
    const int s = e / (words / 4), k = e - s * (words / 4);
    u32x4 out = {0u, 0u, 0u, 0u};
    if (p.mode != 2) {
      const u32x4 ev = first && e == (int)threadIdx.x ? *first : next_e_unit(p, e, toks);
      const float* hrow = nx.h;  // (fetched by tail_prefetch, or by the caller)
      if (p.dtype) {
        const f32x4 h0 = *(const f32x4*)(hrow + 8 * k), h1 = *(const f32x4*)(hrow + 8 * k + 4);
        const float hv[8] = {h0[0], h0[1], h0[2], h0[3], h1[0], h1[1], h1[2], h1[3]};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint16_t lo = silu_bf16(__uint_as_float(ev[w] << 16), hv[2 * w]);
          const uint16_t hi = silu_bf16(__uint_as_float(ev[w] & 0xffff0000u), hv[2 * w + 1]);
          out[w] = (uint32_t)lo | ((uint32_t)hi << 16);
        }
      } else {
        const f32x4 h0 = *(const f32x4*)(hrow + 4 * k);
#pragma unroll
        for (int w = 0; w < 4; ++w) out[w] = __float_as_uint(silu_f32(__uint_as_float(ev[w]), h0[w]));
      }
    }
    *(u32x4*)&nx.u[s * words + 4 * k] = out;
    *(u32x4*)((uint32_t*)p.U + ((size_t)req * p.kk + s) * words + 4 * k) = out;
  }
  lds_barrier();  // (the global copy is read by the next launch only)
}

// Probe logits of the P rows of request `req` at stage d on MFMA: tile t
// (t < 2) holds probes 16 t .. 16 t + 15 as the 16 tokens of a 16x16 tile
// (A: their W rows, staged in nx.pw) against the rows' head inputs in nx.u
// (B), with the same product of absolute values for the margin; waves 2 g + t
// (g < kProbeSplit) take every kProbeSplit-th rank chunk of tile t, and the
// shares are summed.  Two waves per tile measured fastest (eight: their
// sum costs more; one: a 16-chunk chain per wave).  Missing probes get
// kNegBig.
template <int DT>
__device__ void probe_logits(const Plan& p, int P, NextShared& nx) {
  constexpr int KC = DT ? 32 : 16;  // rank elements per MFMA step
  constexpr int ESZ = DT ? 2 : 4;
  constexpr uint32_t kAbs = DT ? 0x7FFF7FFFu : 0x7FFFFFFFu;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nwave = blockDim.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int np = min(kProbe, p.V);
  const int words = p.r * ESZ / 4;
  const int ng = min(nwave / 2, kProbeSplit);  // waves per probe tile
  const int tile = wave & 1, kg = wave >> 1;   // the wave's tile and share of the chunks
  if (kg < ng) {
    const int q = tile * kTile + col;  // the probe this lane's A row holds
    const uint32_t* wrow = nx.pw + q * kProbeRowWords + grp * (KC / 4) * ESZ / 4;
    const uint32_t* urow = nx.u + min(col, P - 1) * words + grp * (KC / 4) * ESZ / 4;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f}, mag = {0.f, 0.f, 0.f, 0.f};
    for (int c = kg; c < p.nchunk; c += ng) {
      const u32x4 a = *(const u32x4*)(wrow + c * KC * ESZ / 4);
      u32x4 b = *(const u32x4*)(urow + c * KC * ESZ / 4);
      if (col >= P) b = u32x4{0u, 0u, 0u, 0u};
      acc = mfma_chunk<DT>(a, b, acc);
      mag = mfma_chunk<DT>(a & kAbs, b & kAbs, mag);
    }
    // the share's C[token 4 grp + i][row col]
    float* pz = nx.pz + (tile * kProbeSplit + kg) * kTile * kTile;
    float* pa = nx.pa + (tile * kProbeSplit + kg) * kTile * kTile;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pz[(4 * grp + i) * kTile + col] = acc[i];
      pa[(4 * grp + i) * kTile + col] = mag[i];
    }
  }
  lds_barrier();
  // the shares summed (in share order); missing probes get kNegBig
  for (int e = threadIdx.x; e < 2 * kTile * kTile; e += blockDim.x) {
    const int t = e / (kTile * kTile), qi = e / kTile, row = e % kTile;  // qi = 16 t + token
    float zs[kProbeSplit], as[kProbeSplit];
#pragma unroll
    for (int g = 0; g < kProbeSplit; ++g) {
      const int gg = min(g, ng - 1);
      zs[g] = nx.pz[(t * kProbeSplit + gg) * kTile * kTile + (qi - t * kTile) * kTile + row];
      as[g] = nx.pa[(t * kProbeSplit + gg) * kTile * kTile + (qi - t * kTile) * kTile + row];
    }
    float z = 0.0f, a = 0.0f;
#pragma unroll
    for (int g = 0; g < kProbeSplit; ++g) {
      if (g < ng) {
        z += zs[g];
        a += as[g];
      }
    }
    if (row < P && qi < np) {
      const bool there = nx.pt[qi] >= 0;
      nx.zl[row * kProbe + qi] = there ? nx.pl[qi] + z : kNegBig;
      nx.al[row * kProbe + qi] = there ? a + fabsf(nx.pl[qi]) : 0.0f;
    }
  }
}

// Bounds tau of the P rows of request `req` at stage d (their head inputs
// in nx.u, the probes in nx.pw / nx.pl / nx.pt): row s gets the k'-th best
// of its logits z = L_d + u_s . W at the probe tokens (distinct tokens, so
// this is at most the row's k'-th best),
// minus a margin of 1e-3 * (1 + sum |terms|), which is far above the float32
// rounding of two r-term sums in any order; with fewer than k' probes the
// bound is -inf.  All threads of the workgroup call it.
__device__ void row_bounds(const Plan& p, int d, int P, int req, NextShared& nx) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nwave = blockDim.x >> 6;
  const int np = min(kProbe, p.V);
  if (p.dtype)
    probe_logits<1>(p, P, nx);
  else
    probe_logits<0>(p, P, nx);
  lds_barrier();
  // two rows per wave: lane 32 h + q holds probe q of row 2 w + h.  A lane
  // whose logit z has fewer than k' probe logits above it and at least k'
  // at or above it holds the k'-th best value (tied lanes write the same).
  const int h = lane >> 5, q = lane & 31;
  for (int s0 = 2 * wave; s0 < P; s0 += 2 * nwave) {
    const int s = min(s0 + h, P - 1);
    const bool live = s0 + h < P && q < np;
    const float z = q < np ? nx.zl[s * kProbe + q] : kNegBig;
    float a = q < np ? nx.al[s * kProbe + q] : 0.0f;
#pragma unroll
    for (int m = 1; m < 32; m <<= 1) a = fmaxf(a, __shfl_xor(a, m));
    f32x4 zv[kProbe / 4];
#pragma unroll
    for (int i = 0; i < kProbe / 4; ++i) zv[i] = *(const f32x4*)(nx.zl + s * kProbe + 4 * i);
    int gt = 0, ge = 0;
#pragma unroll
    for (int k = 0; k < kProbe; ++k) {
      const float o = k < np ? zv[k / 4][k % 4] : -INFINITY;  // (not a probe)
      gt += o > z;
      ge += o >= z;
    }
    if (live && gt < p.kk && ge >= p.kk) p.tau[(size_t)req * P + s] = z - 1e-3f * (1.0f + a);
  }
  lds_barrier();
}

// Multi-launch form: request state in the workspace, the stage-0 head input
// and, when stage 0 runs the wide form, its rows' bounds.  One workgroup
// per request, 16 waves like the merge-and-select workgroups (4 waves made
// the stage-0 bounds 5 us slower per round at 8 requests).
__global__ __launch_bounds__(kSelectThreads) void prologue_kernel(Plan p) {
  __shared__ NextShared nx;
  __shared__ int toks[1];
  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  init_request(p, req, tid, blockDim.x);
  int root = p.root[req];
  if (root < 0 || root >= p.V) root = 0;
  if (tid == 0) {
    p.top_key[(size_t)req * p.N] = node_key(0.0f, 0, root, 0);
    p.top_node[(size_t)req * p.N] = 0;
    p.front_node[req * p.kk] = 0;
    p.front_tok[req * p.kk] = root;
    p.front_score[req * p.kk] = 0.0f;
    toks[0] = root;
  }
  tail_prefetch(p, -1, req, nx);  // depth 0's feature and probes (its state copy is unused)
  __syncthreads();
  next_inputs(p, 0, 1, req, toks, nx);
  if (stage_wide(p.mode, 0, p.R, p.kk) && !p.unbounded) row_bounds(p, 0, 1, req, nx);
}

// After the rows of stage d are in ssh (top-k' children, lse): the stage
// selection of request req (Sec. 4.1, 4.2), the next stage's head input
// and, when the next stage runs the wide form, its rows' bounds.  P is the
// number of head rows of stage d per request.
__device__ void select_tail(const Plan& p, int d, int P, int req, SelShared& ssh, NextShared& nx) {
  const int Pf = d == 0 ? 1 : p.kk;  // frontier size of stage d
  // on the request's state copy in LDS (tail_prefetch, at the kernel's start)
  // (the Shared-Markov and parent-independent modes: the one row of the
  // stage serves every frontier parent of the tree)
  const State st{nx.front_node, nx.front_tok, nx.front_score, nx.top_key, nx.top_node, req};
  // next head input: the new frontier's tokens, or the greedy chain's token
  // (Shared-Markov, known before the selection), or zero
  // (parent-independent); its E loads are issued as soon as the frontier is
  // known and land during the top-N merge
  const bool more = d + 1 < p.B;
  const int Pn = more ? head_rows(p.mode, d + 1, p.kk) : 0;
  __shared__ int chain_tok[1];
  if (p.mode != 0 && threadIdx.x == 0) chain_tok[0] = child_key_token(ssh.rowkeys[0][0]);
  const int* toks = p.mode == 0 ? ssh.next_tok : chain_tok;
  u32x4 ev0 = {0u, 0u, 0u, 0u};
  stage_select_body(p, st, d, Pf, req, 1, ssh, false, p.mode != 0, [&] {
    lds_barrier();
    if (more) ev0 = next_e_first(p, Pn, toks);
  });
  tail_writeback(p, req, nx);
  if (more) {
    next_inputs(p, d + 1, Pn, req, toks, nx, &ev0);
    if (stage_wide(p.mode, d + 1, p.R, p.kk) && !p.unbounded) row_bounds(p, d + 1, Pn, req, nx);
  }
}

// One WG per request: merge the G slice lists of its P rows (waves per row,
// lanes per slice, then xor trees), then the shared stage selection.
template <int KMAX>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(Plan p, int d, int P) {
  constexpr int NW = kSelectThreads / 64;
  __shared__ uint64_t sh_wlist[NW][KMAX];
  __shared__ float2 sh_wms[NW];
  __shared__ SelShared ssh;
  __shared__ NextShared nx;
  const int req = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  tail_prefetch(p, d, req, nx);

  const int wpr = NW / P;  // waves per row
  const int prow = wave / wpr;
  const int sub = wave - prow * wpr;
  uint64_t list[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) list[i] = 0;
  float m = kNegBig, s = 0.0f;
  if (prow < P) {
    const int grow = req * P + prow;
    for (int g = sub * 64 + lane; g < p.G; g += wpr * 64) {
      const size_t o = (size_t)grow * kSlicesMax + g;
      uint64_t other[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) other[i] = p.part_key[o * KMAX + i];
      list_merge(list, other);
      const uint64_t* rec = slice_record(p, 0, grow) + g;
      lse_combine(m, s, child_key_value(rec[0]),
                  __uint_as_float((uint32_t)rec[kHeadKeys * kSlicesMax]));
    }
  }
#pragma unroll
  for (int mask = 1; mask < 64; mask <<= 1) {
    list_merge_xor(list, mask);
    lse_combine_xor(m, s, mask);
  }
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) sh_wlist[wave][i] = list[i];
    sh_wms[wave] = make_float2(m, s);
  }
  __syncthreads();
  if (prow < P && sub == 0) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) list[i] = lane < wpr ? sh_wlist[wave + lane][i] : 0;
    m = lane < wpr ? sh_wms[wave + lane].x : kNegBig;
    s = lane < wpr ? sh_wms[wave + lane].y : 0.0f;
#pragma unroll
    for (int mask = 1; mask < 16; mask <<= 1) {
      list_merge_xor(list, mask);
      lse_combine_xor(m, s, mask);
    }
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) ssh.rowkeys[prow][i] = list[i];
      ssh.lse[prow] = m + logf(s);
    }
  }
  __syncthreads();
  select_tail(p, d, P, req, ssh, nx);
}

constexpr int kWideWaves = 8;       // waves of a wide head workgroup
constexpr int kThrRows = kWideWaves * kTile;  // rows of one column group: 8 blocks of 16
constexpr int kThrSlots = 4;        // super-tiles (two W tiles) in the LDS ring
constexpr int kLUnits = 64;         // 16-byte units of L_d per ring slot (one load instruction)
constexpr int kLWave = 7;           // the wave that loads L_d into the ring

// LDS of head_thr_kernel.  The ring slots are separate objects, so that the
// compiler can tell the slot being loaded from the one being read (a load
// into LDS that might alias a read would make it wait for every load in
// flight); slot 0 also serves the exact path's list merges.
template <int NCMAX, int KMAX>
struct ThrShape {
  static constexpr int kSlot = 2 * kTile * (4 * NCMAX + 1);      // u32x4: 32 padded W rows
  static constexpr int kScratch = kWideWaves * kTile * KMAX / 2;  // u32x4 of the merges
  static constexpr int kSlot0 = kSlot > kScratch ? kSlot : kScratch;
};

// B fragments of one frontier row (its head input; zero past the rank and
// for rows past the stage's).
template <int DT, int NCMAX>
__device__ __forceinline__ void load_urow(const Plan& p, int P, int row, bool ok, int lg,
                                          u32x4 (&b)[NCMAX]) {
  constexpr int KC = DT ? 32 : 16;
  constexpr int ESZ = DT ? 2 : 4;
  const int req = ok ? row / P : 0, slot = ok ? row - req * P : 0;
  const char* u = (const char*)p.U + ((size_t)(req * p.kk + slot) * p.r + lg * (KC / 4)) * ESZ;
#pragma unroll
  for (int c = 0; c < NCMAX; ++c) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (c < p.nchunk && ok) v = *(const u32x4*)(u + (size_t)c * KC * ESZ);
    b[c] = v;
  }
}

// The careful path for one row's four logits of a tile (tokens tb .. tb+3):
// online (max, sum of exp) with rescaling, and every logit at or above tau
// appended to the row's candidates (a count past KMAX marks an overflow).
template <int KMAX>
__device__ __forceinline__ void thr_row_slow(const Plan& p, const float (&z)[4], int tb, float& m,
                                             float& s, float tau, uint64_t* cand, int* cnt) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (tb + i < p.V) {
      const float v = z[i];
      if (v > m) {
        s *= exp2_raw((m - v) * kLog2e);
        m = v;
      }
      s += exp2_raw((v - m) * kLog2e);
      if (v >= tau) {
        const int slot = atomicAdd(cnt, 1);
        if (slot < KMAX) cand[slot] = child_key(v, tb + i);
      }
    }
  }
}

// The exact path of a slice for rows whose candidates overflowed (more than
// KMAX at or above the bound): the slice is streamed again for those rows, 16
// at a time, with full per-lane top-KMAX lists, and each row's KMAX best keys
// are published.  All threads of the workgroup call it.
template <int DT, int NCMAX, int KMAX>
__device__ __forceinline__ void thr_exact(const Plan& p, int d, int P, int slice, int t0, int t1, const int* ovl,
                          int nov, uint64_t* scratch) {
  const int wave = threadIdx.x >> 6;
  for (int b = 0; b < nov; b += kTile) {
    HeadLane h(p, P, 0);  // lane geometry; its row is the b + col-th listed one
    const bool ok = b + h.col < nov;
    const int row = ok ? ovl[b + h.col] : 0;
    h.row = row;
    h.row_ok = h.b_ok = ok;
    h.req = h.b_req = row / P;
    h.slot = h.b_slot = row - h.req * P;
    u32x4 bf[NCMAX];
    load_urow<DT, NCMAX>(p, P, row, ok, h.grp, bf);
    RowAcc<KMAX> ra;
    ra.init();
    for (int t = t0 + wave; t < t1; t += kWideWaves) {
      u32x4 a[NCMAX];
      uint32_t l[4];
      load_afrag<DT, NCMAX>(p, h, t, a);
      load_lfrag<DT>(p, h, d, t, l);
      tile_step<DT, NCMAX, KMAX>(p, h, a, bf, l, t, ra);
    }
    list_merge_pair<16>(ra.list);
    list_merge_pair<32>(ra.list);
    if (h.grp == 0) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) scratch[(i * kWideWaves + wave) * kTile + h.col] = ra.list[i];
    }
    __syncthreads();
    if (wave == 0 && h.grp == 0 && ok) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) ra.list[i] = scratch[i * kWideWaves * kTile + h.col];
      for (int w = 1; w < kWideWaves; ++w) {
        uint64_t o[KMAX];
#pragma unroll
        for (int i = 0; i < KMAX; ++i) o[i] = scratch[(i * kWideWaves + w) * kTile + h.col];
        list_merge(ra.list, o);
      }
      const size_t o = (size_t)row * kSlicesMax + slice;
#pragma unroll
      for (int i = 0; i < KMAX; ++i) p.part_key[o * KMAX + i] = ra.list[i];
      p.thr_cnt[o] = KMAX;
    }
    __syncthreads();
  }
}

// 16 bytes per lane from global memory straight into LDS (lane l's bytes at
// lds_dst + 16 l), counted in vmcnt like any vector-memory load.  Issued as
// inline assembly: the compiler does not see the LDS write, so it does not
// make later LDS reads wait for every load in flight (it cannot tell ring
// slots apart); the kernel orders them itself with wait_vmcnt and a
// barrier.  M0 holds the LDS base; nothing else in the kernels that use it
// keeps a value in M0 across it.
__device__ __forceinline__ void load_lds16(const void* src, const void* lds_dst) {
  const uint32_t base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_dst);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(base)
               : "memory", "m0");
}

// s_waitcnt with only the vector-memory count limited (gfx9 encoding:
// vmcnt bits 3:0 and 15:14, expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// One V-slice for up to 128 frontier rows of a wide stage.  Wave w multiplies
// tile (2 s + w / 4) of super-tile s into the two 16-row column blocks
// 2 (w % 4) and 2 (w % 4) + 1 of its column group (their head inputs stay in
// registers), so each W tile read from LDS serves 32 rows, and the 8 waves
// take two tiles per step.  W goes from memory straight into a ring of
// kThrSlots super-tiles in LDS (16 bytes per lane, already in MFMA fragment
// order), kThrSlots - 1 super-tiles ahead, with the lanes' L_d values in a
// register ring alongside; a step waits for its own loads (counted), then
// for the other waves' at the barrier.  Per row the workgroup publishes its
// slice's (max, sum of exp) and the logits at or above the row's bound tau
// (at most KMAX; a row with more takes the exact path).  The grid has
// 8 * ceil(G / 8) * (column groups) workgroups, XCD-ordered as in head_kernel.
template <int DT, int NCMAX, int KMAX>
__global__ __launch_bounds__(kWideWaves * 64) void head_thr_kernel(Plan p, int d, int P) {
  using SH = ThrShape<NCMAX, KMAX>;
  constexpr int KC = DT ? 32 : 16;
  constexpr int ESZ = DT ? 2 : 4;
  // loads per wave per super-tile: 32 rows of at most 4 NCMAX <= 64 units
  // each, one instruction per row, over the 8 waves
  constexpr int CPW = 2 * kTile / kWideWaves;
  static_assert(4 * NCMAX <= 64, "a W row must fit one load instruction");
  constexpr int LW = DT ? 2 : 4;     // 32-bit words of L_d per row and tile per lane
  constexpr int GROUP = CPW + 2;     // vector-memory instructions per super-tile per wave
  typedef uint32_t lvec __attribute__((ext_vector_type(LW)));
  __shared__ u32x4 ring0[SH::kSlot0], ring1[SH::kSlot], ring2[SH::kSlot], ring3[SH::kSlot];
  __shared__ u32x4 lslot[kThrSlots][kLUnits];  // L_d of the group's requests per super-tile
  __shared__ uint64_t cand[kThrRows * KMAX];  // each row's candidates
  __shared__ int ccnt[kThrRows];              // their count (past KMAX: overflow)
  __shared__ float2 msx[kThrRows];            // the second wave's row statistics
  __shared__ int ovl[kThrRows + 1];           // rows for the exact path, and their count
  // (a switch over a constant after unrolling: the objects stay distinct)
  auto slot_ptr = [&](int slot) -> u32x4* {
    switch (slot) {
      case 0: return ring0;
      case 1: return ring1;
      case 2: return ring2;
      default: return ring3;
    }
  };

  const int rows = p.R * P;
  const int ncb = (rows + kTile - 1) / kTile;
  const int ngrp = (ncb + kWideWaves - 1) / kWideWaves;
  const int x = blockIdx.x & 7, jb = blockIdx.x >> 3;
  const int grp = jb % ngrp;
  const int slice = (jb / ngrp) * 8 + x;
  if (slice >= p.G) return;  // the whole workgroup
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int pair = wave & 3, half = wave >> 2;
  const int col = lane & 15, lg = lane >> 4;
  const int row0 = grp * kThrRows;
  const int lr0 = 2 * pair * kTile + col, lr1 = lr0 + kTile;  // rows within the group
  const int gr0 = row0 + lr0, gr1 = row0 + lr1;
  const bool ok0 = gr0 < rows, ok1 = gr1 < rows;
  const bool live = row0 + 2 * pair * kTile < rows;  // the wave has a row to compute
  const int q0 = ok0 ? gr0 / P : 0, q1 = ok1 ? gr1 / P : 0;  // requests of the two rows
  // L_d goes through the ring (as W does) when the group's requests fit one
  // load instruction per super-tile and their rows are 16-byte aligned;
  // otherwise each lane loads its own L_d words into registers
  constexpr int TPU = 16 / ESZ;            // tokens per 16-byte unit
  constexpr int UPR = 2 * kTile / TPU;     // units of one request's row per super-tile
  const int q_lo = row0 / P;
  const int nq = (min(row0 + kThrRows, rows) - 1) / P - q_lo + 1;
  const bool lds_l = nq * UPR <= kLUnits && p.V % TPU == 0 && p.V >= 2 * kTile &&
                     ((uintptr_t)p.L & 15) == 0;
  const int j0 = min(max(q0 - q_lo, 0), nq - 1), j1 = min(max(q1 - q_lo, 0), nq - 1);

  if (blockIdx.x == 0) TIMELINE_STAMP(3, d, 0);
  for (int i = tid; i < kThrRows; i += blockDim.x) ccnt[i] = 0;
  if (tid == 0) ovl[kThrRows] = 0;

  // per row: bound, running max and sum; thr = min(tau, m) decides the careful
  // path (rows past the stage's never take it)
  const float big = 3.0e38f;
  float tau0 = ok0 ? (p.unbounded ? kNegBig : p.tau[gr0]) : big;
  float tau1 = ok1 ? (p.unbounded ? kNegBig : p.tau[gr1]) : big;
  float m0 = ok0 ? tau0 : kNegBig, s0 = 0.0f;
  float m1 = ok1 ? tau1 : kNegBig, s1 = 0.0f;
  float thr0 = ok0 ? fminf(tau0, m0) : big, thr1 = ok1 ? fminf(tau1, m1) : big;

  const int t0 = slice * p.tiles_per_slice;
  const int t1 = min(t0 + p.tiles_per_slice, p.ntiles);
  const int nsup = (t1 - t0 + 1) / 2;
  const int ru = p.r * ESZ / 16;  // 16-byte units of a W row (a multiple of 4, at most 64)
  const char* lrow0 = (const char*)p.L + ((size_t)q0 * p.B + d) * p.V * ESZ;
  const char* lrow1 = (const char*)p.L + ((size_t)q1 * p.B + d) * p.V * ESZ;
  // whether 16-bit L_d rows allow one aligned vector load of four tokens
  const bool lvec_ok = ((size_t)p.V * ESZ) % (LW * 4) == 0;

  // One super-tile's loads: its 32 token rows of W straight into its ring
  // slot, one row per instruction (lane l loads the row's l-th 16 bytes, so
  // an instruction reads one contiguous run), then the lane's L_d words for
  // both rows.  In the slot, row i starts at unit i (ru + 1): the one unit of
  // padding puts the 16 rows of an MFMA A-fragment read (one unit each) in 16
  // different bank groups.  Tokens past the slice or V re-read the last one.
  // (slot == s % kThrSlots, passed as a constant of the unrolled loops)
  // (LL: L_d goes through the ring; otherwise into the lane's registers)
  auto issue = [&](auto ll, int s, int slot, lvec (&l)[2]) __attribute__((always_inline)) {
    constexpr bool LL = decltype(ll)::value;
#pragma unroll
    for (int q = 0; q < CPW; ++q) {
      const int row = wave + q * kWideWaves;  // token row of the super-tile
      const int t = min(t0 + 2 * s + row / kTile, t1 - 1);
      const int tok = min(t * kTile + (row & (kTile - 1)), p.V - 1);
      const char* src = (const char*)p.Wt + (size_t)tok * p.r * ESZ + (size_t)min(lane, ru - 1) * 16;
      if (lane < ru) load_lds16(src, slot_ptr(slot) + row * (ru + 1));
    }
    if constexpr (LL) {
      // one wave loads every request's L_d words of the super-tile: lane l
      // takes unit l % UPR of request l / UPR (lanes past the requests
      // repeat the last one; units past V re-read the row's last unit)
      if (wave == kLWave) {
        const int j = min(lane / UPR, nq - 1), u = lane - (lane / UPR) * UPR;
        const int tk = min((t0 + 2 * s) * kTile + u * TPU, p.V - TPU);
        load_lds16((const char*)p.L + (((size_t)(q_lo + j) * p.B + d) * p.V + tk) * ESZ,
                   &lslot[slot][0]);
      }
    } else {
      const int t = min(t0 + 2 * s + half, t1 - 1);
      const int tb = min(t * kTile + lg * 4, p.V - 4 > 0 ? p.V - 4 : 0);
      if (lvec_ok && p.V >= 4) {
        l[0] = *(const lvec*)(lrow0 + (size_t)tb * ESZ);
        l[1] = *(const lvec*)(lrow1 + (size_t)tb * ESZ);
      } else {  // (unaligned rows: word by word)
        lvec a, b;
#pragma unroll
        for (int i = 0; i < LW; ++i) { a[i] = 0u; b[i] = 0u; }
        const int tb2 = t * kTile + lg * 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = min(tb2 + i, p.V - 1);
          const uint32_t ra = load_raw<DT>(p.L, ((size_t)q0 * p.B + d) * p.V + v);
          const uint32_t rb = load_raw<DT>(p.L, ((size_t)q1 * p.B + d) * p.V + v);
          if (DT) {
            a[i / 2] |= ra << (16 * (i & 1));
            b[i / 2] |= rb << (16 * (i & 1));
          } else {
            a[i] = ra;
            b[i] = rb;
          }
        }
        l[0] = a;
        l[1] = b;
      }
    }
  };
  // the four L_d values of the lane's tokens (tokens tb .. tb + 3 of its
  // tile, realigned when a register vector load had to start earlier)
  auto lval = [&](auto ll, const lvec& l, int tb, int i) __attribute__((always_inline)) -> float {
    constexpr bool LL = decltype(ll)::value;
    const int shift = (!LL && lvec_ok && p.V >= 4) ? tb - min(tb, p.V - 4 > 0 ? p.V - 4 : 0) : 0;
    const int e = min(i + shift, 3);
    return DT ? __uint_as_float((e & 1) ? (l[e / 2] & 0xffff0000u) : (l[e / 2] << 16))
              : __uint_as_float(l[e]);
  };

  // the head inputs of the wave's rows (B fragments) and the bounds first,
  // waited for at once: with no compiler-issued load in flight, the
  // compiler puts no wait of its own into the ring loop (it cannot count
  // the ring's loads, so any wait it placed there would drain the whole
  // ring).  The register path's L_d loads do get such waits; it serves
  // only groups with many requests or unaligned rows.
  // The 128 rows' head inputs go through the idle ring first, each row
  // loaded once (row i of the group into ring slot i / 32, at the W rows'
  // padded stride, so that wave pair q's 32 rows fill slot q): the two
  // waves of a pair then read the same rows from LDS instead of both
  // fetching them.  Rows past the stage's re-read a valid one and read back
  // as zero.
  u32x4 b0[NCMAX], b1[NCMAX];
  {
    constexpr int RPW = kThrRows / kWideWaves;  // rows per wave
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
      const int i = wave + k * kWideWaves;  // row of the group
      const int gr = min(row0 + i, rows - 1);
      const int req = gr / P, slot = gr - req * P;
      const char* src = (const char*)p.U + ((size_t)(req * p.kk + slot) * p.r) * ESZ +
                        (size_t)min(lane, ru - 1) * 16;
      if (lane < ru) load_lds16(src, slot_ptr(i / (2 * kTile)) + (i % (2 * kTile)) * (ru + 1));
    }
    wait_vmcnt<0>();
    __syncthreads();
    const u32x4* us = slot_ptr(pair) + col * (ru + 1) + lg;
#pragma unroll
    for (int c = 0; c < NCMAX; ++c) {
      const u32x4 v0 = us[c * 4], v1 = us[kTile * (ru + 1) + c * 4];
      const bool in = c < p.nchunk && live;
      b0[c] = in && ok0 ? v0 : u32x4{0u, 0u, 0u, 0u};
      b1[c] = in && ok1 ? v1 : u32x4{0u, 0u, 0u, 0u};
    }
    __syncthreads();  // (the prefetch below overwrites the ring)
  }

  auto stream = [&](auto ll) __attribute__((always_inline)) {
    constexpr bool LL = decltype(ll)::value;
    // the first super-tiles' loads; the barrier also makes the candidate
    // counts zero for every wave before any appends
    lvec lring[kThrSlots][2];
#pragma unroll
    for (int i = 0; i + 1 < kThrSlots; ++i)
      if (i < nsup) issue(ll, i, i, lring[i]);
    __syncthreads();
    // vector-memory instructions per super-tile of this wave
    const bool extra = LL && wave == kLWave;
    for (int sb = 0; sb < nsup; sb += kThrSlots) {
#pragma unroll
      for (int i = 0; i < kThrSlots; ++i) {
        const int s = sb + i;
        if (s >= nsup) break;
        // this wave's loads of super-tile s (and of its L_d words) have
        // landed once at most the later super-tiles' loads are outstanding
        const int ahead = min(nsup - 1 - s, kThrSlots - 2);
        constexpr int G0 = LL ? CPW : GROUP;
        if (ahead == 0)
          wait_vmcnt<0>();
        else if (!extra)
          ahead == 2 ? wait_vmcnt<2 * G0>() : wait_vmcnt<G0>();
        else
          ahead == 2 ? wait_vmcnt<2 * G0 + 2>() : wait_vmcnt<G0 + 1>();
        // and every wave's: ring slot s is complete, slot s - 1 is free
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (s + kThrSlots - 1 < nsup)
          issue(ll, s + kThrSlots - 1, (i + kThrSlots - 1) % kThrSlots,
                lring[(i + kThrSlots - 1) % kThrSlots]);
        const int t = t0 + 2 * s + half;
        if (live && t < t1) {
          f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
          // lane: token col of tile `half`, units c * 4 + lg (a row's units
          // past its rank, up to 4 NCMAX, still lie inside the ring slot)
          const u32x4* a = slot_ptr(i) + (half * kTile + col) * (ru + 1) + lg;  // (s % kThrSlots == i)
          if constexpr (LL) {
            // A fragments in groups of AG, the next group's reads in flight
            // while this group's MFMAs run (one read at a time would pay the
            // LDS latency per chunk); the scheduling barriers keep that order
            // Chunks past the rank (c >= nchunk) are read at their constant
            // offsets, which stay inside the slot, and skipped: the reads
            // then need no address register per chunk.
            constexpr int AG = NCMAX >= 16 ? 2 : 4, NG = (NCMAX + AG - 1) / AG;
            u32x4 ag[2][AG];
#pragma unroll
            for (int e = 0; e < AG; ++e) ag[0][e] = a[min(e, NCMAX - 1) * 4];
#pragma unroll
            for (int g = 0; g < NG; ++g) {
              if (g + 1 < NG) {
#pragma unroll
                for (int e = 0; e < AG; ++e)
                  ag[(g + 1) & 1][e] = a[min((g + 1) * AG + e, NCMAX - 1) * 4];
              }
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int e = 0; e < AG; ++e) {
                const int c = g * AG + e;
                if (c < NCMAX && c < p.nchunk) {
                  c0 = mfma_chunk<DT>(ag[g & 1][e], b0[c], c0);
                  c1 = mfma_chunk<DT>(ag[g & 1][e], b1[c], c1);
                }
              }
              __builtin_amdgcn_sched_barrier(0);
            }
          } else {
#pragma unroll
            for (int c = 0; c < NCMAX; ++c) {
              const u32x4 av = a[c * 4];
              if (c < p.nchunk) {
                c0 = mfma_chunk<DT>(av, b0[c], c0);
                c1 = mfma_chunk<DT>(av, b1[c], c1);
              }
            }
          }
          const int tb = t * kTile + lg * 4;
          lvec la, lb;
          if constexpr (LL) {  // the rows' requests' L_d words of the lane's four tokens
            const char* lo = (const char*)&lslot[i][0] + (half * kTile + lg * 4) * ESZ;
            la = *(const lvec*)(lo + j0 * UPR * 16);
            lb = *(const lvec*)(lo + j1 * UPR * 16);
          } else {
            la = lring[i][0];
            lb = lring[i][1];
          }
          float z0[4], z1[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            z0[e] = c0[e] + lval(ll, la, tb, e);
            z1[e] = c1[e] + lval(ll, lb, tb, e);
          }
          const float mx0 = fmaxf(fmaxf(z0[0], z0[1]), fmaxf(z0[2], z0[3]));
          const float mx1 = fmaxf(fmaxf(z1[0], z1[1]), fmaxf(z1[2], z1[3]));
          // the careful path: a logit at or above the bound or the running
          // maximum, or tokens past V (only in the vocabulary's last tile)
          const bool hot = mx0 >= thr0 || mx1 >= thr1 || tb + 3 >= p.V;
          if (__builtin_expect(__any(hot), 0)) {
            if (ok0) thr_row_slow<KMAX>(p, z0, tb, m0, s0, tau0, cand + lr0 * KMAX, ccnt + lr0);
            if (ok1) thr_row_slow<KMAX>(p, z1, tb, m1, s1, tau1, cand + lr1 * KMAX, ccnt + lr1);
            thr0 = ok0 ? fminf(tau0, m0) : big;
            thr1 = ok1 ? fminf(tau1, m1) : big;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              s0 += exp2_raw((z0[e] - m0) * kLog2e);
              s1 += exp2_raw((z1[e] - m1) * kLog2e);
            }
          }
        }
      }
    }
  };
  if (lds_l)
    stream(std::true_type{});
  else
    stream(std::false_type{});
  __syncthreads();  // the ring is free for the exact path; candidates complete
  if (blockIdx.x == 0) TIMELINE_STAMP(3, d, 1);

  // the row statistics: the four lane groups, then the two waves of a row
  lse_combine_pair<16>(m0, s0);
  lse_combine_pair<32>(m0, s0);
  lse_combine_pair<16>(m1, s1);
  lse_combine_pair<32>(m1, s1);
  if (half == 1 && lg == 0) {
    msx[lr0] = make_float2(m0, s0);
    msx[lr1] = make_float2(m1, s1);
  }
  __syncthreads();
  if (half == 0 && lg == 0) {
    if (ok0) {
      lse_combine(m0, s0, msx[lr0].x, msx[lr0].y);
      *(float2*)(p.thr_ms + ((size_t)gr0 * kSlicesMax + slice) * 2) = make_float2(m0, s0);
    }
    if (ok1) {
      lse_combine(m1, s1, msx[lr1].x, msx[lr1].y);
      *(float2*)(p.thr_ms + ((size_t)gr1 * kSlicesMax + slice) * 2) = make_float2(m1, s1);
    }
  }
  // the candidates: rows within KMAX publish theirs, the others are listed
  // for the exact path
  for (int e = tid; e < kThrRows * KMAX; e += blockDim.x) {
    const int lr = e / KMAX, i = e - lr * KMAX;
    const int gr = row0 + lr;
    if (gr < rows) {
      const int c = ccnt[lr];
      const size_t o = (size_t)gr * kSlicesMax + slice;
      if (c <= KMAX) {
        if (i < c) p.part_key[o * KMAX + i] = cand[lr * KMAX + i];
        if (i == 0) p.thr_cnt[o] = c;
      } else if (i == 0) {
        ovl[atomicAdd(&ovl[kThrRows], 1)] = gr;
      }
    }
  }
  __syncthreads();
  const int nov = ovl[kThrRows];
  if (nov > 0)
    thr_exact<DT, NCMAX, KMAX>(p, d, P, slice, t0, t1, ovl, nov, (uint64_t*)ring0);
  if (blockIdx.x == 0) TIMELINE_STAMP(3, d, 2);
}

// One WG per request after a wide head stage: each of its rows (one wave per
// row) merges the slices' (max, sum of exp) into its lse and the slices'
// candidates into its k' children; then the stage selection, the next
// stage's head input and its rows' bounds (select_tail).
constexpr int kMergeCap = 256;  // candidates of a row ranked in LDS (more: list merges)

template <int KMAX>
__global__ __launch_bounds__(kSelectThreads) void mergesel_kernel(Plan p, int d, int P) {
  __shared__ SelShared ssh;
  __shared__ NextShared nx;
  __shared__ __attribute__((aligned(16))) uint64_t mk[kNarrowRows][kMergeCap];
  __shared__ int msrc[kNarrowRows][kMergeCap];  // where each gathered key comes from
  const int req = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (req == 0) TIMELINE_STAMP(4, d, 0);
  // the lane's slices of its wave's row (at most kSlicesMax / 64):
  // statistics and counts first, all loads in flight together, then the
  // state and next-stage loads behind them, then the few candidates
  constexpr int SPL = kSlicesMax / 64;
  const int gr = req * P + min(wave, P - 1);
  float2 v[SPL];
  int c[SPL];
  if (wave < P) {
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      const int g = lane + 64 * i;
      const size_t o = (size_t)gr * kSlicesMax + min(g, p.G - 1);
      v[i] = *(const float2*)(p.thr_ms + o * 2);
      c[i] = g < p.G ? min(p.thr_cnt[o], KMAX) : 0;
    }
  }
  tail_prefetch(p, d, req, nx);
  if (wave < P) {
    float m = kNegBig, s = 0.0f;
    int mine = 0;
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      if (lane + 64 * i < p.G) lse_combine(m, s, v[i].x, v[i].y);
      mine += c[i];
    }
    const float M = wave_max_f32(m);
    const float S = wave_sum_f32(s * exp2_raw((m - M) * kLog2e));
    // the row's candidates, gathered in LDS at the lanes' exclusive prefix sums
    int off = mine;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
      const int o = __shfl_up(off, sh);
      if (lane >= sh) off += o;
    }
    const int n = __shfl(off, 63);
    off -= mine;
    uint64_t* keys = mk[wave];
    if (n <= kMergeCap) {
      // first where each key sits (LDS stores only), then every key's load
      // in flight at once: a load per key in turn would pay its latency
      // once per candidate
      int* src = msrc[wave];
#pragma unroll
      for (int i = 0; i < SPL; ++i)
        for (int j = 0; j < c[i]; ++j) src[off++] = (lane + 64 * i) * KMAX + j;
      __builtin_amdgcn_wave_barrier();
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      const uint64_t* rk = p.part_key + (size_t)gr * kSlicesMax * KMAX;
      uint64_t kv[kMergeCap / 64];
#pragma unroll
      for (int t = 0; t < kMergeCap / 64; ++t) {
        const int e = lane + 64 * t;
        kv[t] = e < n ? rk[src[e]] : 0;
      }
#pragma unroll
      for (int t = 0; t < kMergeCap / 64; ++t)
        if (lane + 64 * t < n) keys[lane + 64 * t] = kv[t];
    }
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (n <= kMergeCap) {
      // rank each key among the row's (keys are unique: distinct tokens)
      if (lane < KMAX) ssh.rowkeys[wave][lane] = 0;
      __builtin_amdgcn_wave_barrier();
      for (int k = lane; k < n; k += 64) {
        const uint64_t key = keys[k];
        const int rank = count_greater(keys, n, key);
        if (rank < KMAX) ssh.rowkeys[wave][rank] = key;
      }
    } else {
      // (many candidates: per-lane top-KMAX lists merged over the wave)
      uint64_t lst[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) lst[i] = 0;
#pragma unroll
      for (int i = 0; i < SPL; ++i) {
        const size_t o = (size_t)gr * kSlicesMax + min(lane + 64 * i, p.G - 1);
        for (int j = 0; j < c[i]; ++j) {
          const uint64_t k = p.part_key[o * KMAX + j];
          if (k > lst[KMAX - 1]) list_insert(lst, k);
        }
      }
#pragma unroll
      for (int mask = 1; mask < 64; mask <<= 1) list_merge_xor(lst, mask);
      if (lane == 0) {
#pragma unroll
        for (int i = 0; i < KMAX; ++i) ssh.rowkeys[wave][i] = lst[i];
      }
    }
    if (lane == 0) ssh.lse[wave] = M + logf(S);
  }
  __syncthreads();
  if (req == 0) TIMELINE_STAMP(4, d, 1);
  select_tail(p, d, P, req, ssh, nx);
  if (req == 0) TIMELINE_STAMP(4, d, 2);
}

// Zero the words the persistent round polls (slice partials of every stage,
// row and slice, and the frontier words) and mark every request as not built.
__global__ __launch_bounds__(256) void clear_kernel(Plan p) {
  const int per = p.kmax + kRecWords;  // list words, then record words
  const int nrec = p.stages * p.rows_max * p.G;
  const int n = nrec * per;
  const int stride = gridDim.x * blockDim.x;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int rec = i / per, w = i - rec * per;
    const int sr = rec / p.G, slice = rec - sr * p.G;  // (stage, row), slice
    if (w < p.kmax)
      p.part_key[((size_t)sr * kSlicesMax + slice) * p.kmax + w] = 0;
    else
      p.part_hd[((size_t)sr * kRecWords + (w - p.kmax)) * kSlicesMax + slice] = 0;
  }
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < p.stages * p.rows_max; i += stride)
    p.front_w[i] = 0;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < p.R; i += stride) p.o_count[i] = -1;
}

__global__ __launch_bounds__(kEmitThreads) void emit_kernel(Plan p) {
  emit_request(p, global_state(p), blockIdx.x);
}

__global__ __launch_bounds__(kMaskThreads) void mask_kernel(const int* parent, const int* count,
                                                            int N, uint32_t* mask) {
  __shared__ int sh_par[PCTREE_MASK_MAX_N];
  __shared__ uint32_t sh_words[kMaskThreads * (PCTREE_MASK_MAX_N / 32)];
  const int req = blockIdx.x;
  for (int i = threadIdx.x; i < N; i += blockDim.x) sh_par[i] = parent[(size_t)req * N + i];
  __syncthreads();
  const int c = min(max(count[req], 0), N);
  mask_rows(sh_par, c, N, mask + (size_t)req * N * ((N + 31) / 32), sh_words,
            PCTREE_MASK_MAX_N / 32);
}

// ---------------------------------------------------------------------------
// dispatch
// ---------------------------------------------------------------------------
typedef void (*StageFn)(Plan, int, int);
typedef void (*RoundFn)(Plan);

#define PCTREE_KMAX_SWITCH(KERNEL, DT, NCMAX, kmax) \
  switch (kmax) {                                   \
    case 1: return KERNEL<DT, NCMAX, 1>;            \
    case 2: return KERNEL<DT, NCMAX, 2>;            \
    case 4: return KERNEL<DT, NCMAX, 4>;            \
    case 8: return KERNEL<DT, NCMAX, 8>;            \
    default: return KERNEL<DT, NCMAX, 16>;          \
  }

// round kernels: KMAX up to 16 without fold, up to 8 with it
#define PCTREE_ROUND_KMAX_SWITCH(KERNEL, DT, NCMAX, kmax, FOLD)        \
  if (FOLD) {                                                         \
    switch (kmax) {                                                   \
      case 1: return KERNEL<DT, NCMAX, 1, true>;                      \
      case 2: return KERNEL<DT, NCMAX, 2, true>;                      \
      case 4: return KERNEL<DT, NCMAX, 4, true>;                      \
      default: return KERNEL<DT, NCMAX, 8, true>;                     \
    }                                                                 \
  }                                                                   \
  switch (kmax) {                                                     \
    case 1: return KERNEL<DT, NCMAX, 1, false>;                       \
    case 2: return KERNEL<DT, NCMAX, 2, false>;                       \
    case 4: return KERNEL<DT, NCMAX, 4, false>;                       \
    case 8: return KERNEL<DT, NCMAX, 8, false>;                       \
    default: return KERNEL<DT, NCMAX, 16, false>;                     \
  }

#define PCTREE_DISPATCH(KERNEL, p)                                    \
  if ((p).dtype) {                                                    \
    if ((p).nchunk <= 4) { PCTREE_KMAX_SWITCH(KERNEL, 1, 4, (p).kmax) } \
    if ((p).nchunk <= 8) { PCTREE_KMAX_SWITCH(KERNEL, 1, 8, (p).kmax) } \
    if ((p).nchunk <= 12) { PCTREE_KMAX_SWITCH(KERNEL, 1, 12, (p).kmax) } \
    PCTREE_KMAX_SWITCH(KERNEL, 1, 16, (p).kmax)                       \
  }                                                                   \
  if ((p).nchunk <= 2) { PCTREE_KMAX_SWITCH(KERNEL, 0, 2, (p).kmax) } \
  PCTREE_KMAX_SWITCH(KERNEL, 0, 8, (p).kmax)

StageFn head_fn(const Plan& p) { PCTREE_DISPATCH(head_kernel, p) }
StageFn head_thr_fn(const Plan& p) { PCTREE_DISPATCH(head_thr_kernel, p) }

// NCMAX of the instantiation PCTREE_DISPATCH picks.
int nchunk_max(const Plan& p) {
  if (p.dtype) return p.nchunk <= 4 ? 4 : (p.nchunk <= 8 ? 8 : (p.nchunk <= 12 ? 12 : 16));
  return p.nchunk <= 2 ? 2 : 8;
}
// The folded form serves rounds whose stages have at most 8 frontier rows.
bool round_fold(const Plan& p) { return p.R * p.kk <= 8; }

RoundFn round_fn(const Plan& p) {
  const bool fold = round_fold(p);
  if (p.dtype) {
    if (p.nchunk <= 4) { PCTREE_ROUND_KMAX_SWITCH(round_kernel, 1, 4, p.kmax, fold) }
    if (p.nchunk <= 8) { PCTREE_ROUND_KMAX_SWITCH(round_kernel, 1, 8, p.kmax, fold) }
    if (p.nchunk <= 12) { PCTREE_ROUND_KMAX_SWITCH(round_kernel, 1, 12, p.kmax, fold) }
    PCTREE_ROUND_KMAX_SWITCH(round_kernel, 1, 16, p.kmax, fold)
  }
  if (p.nchunk <= 2) { PCTREE_ROUND_KMAX_SWITCH(round_kernel, 0, 2, p.kmax, fold) }
  PCTREE_ROUND_KMAX_SWITCH(round_kernel, 0, 8, p.kmax, fold)
}

StageFn mergesel_fn(int kmax) {
  switch (kmax) {
    case 1: return mergesel_kernel<1>;
    case 2: return mergesel_kernel<2>;
    case 4: return mergesel_kernel<4>;
    case 8: return mergesel_kernel<8>;
    default: return mergesel_kernel<16>;
  }
}

StageFn select_fn(int kmax) {
  switch (kmax) {
    case 1: return select_kernel<1>;
    case 2: return select_kernel<2>;
    case 4: return select_kernel<4>;
    case 8: return select_kernel<8>;
    default: return select_kernel<16>;
  }
}

// Call tags: 1 .. kTagMask in turn (0 is what the clear leaves).
uint32_t next_tag() {
  static std::atomic<uint32_t> seq{0};
  return seq.fetch_add(1, std::memory_order_relaxed) % kTagMask + 1;
}

// Per-device facts for the persistent launch, queried once per device.
struct DeviceInfo {
  int cus = 0;
  long long ticks_per_s = 0;
};

DeviceInfo device_info() {
  static DeviceInfo cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DeviceInfo{};
  DeviceInfo& di = cache[dev];
  if (di.cus == 0) {
    int cus = 0, khz = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) khz = 0;
    di.ticks_per_s = (long long)(khz > 0 ? khz : 100000) * 1000;
    di.cus = cus;
  }
  return di;
}

}  // namespace

DebugConfig& debug_config() {
  static DebugConfig cfg;
  return cfg;
}

hipError_t launch_round(const Plan& p0, hipStream_t st) {
  const DebugConfig dbg = debug_config();
  const bool narrow = p0.R * p0.kk <= kNarrowRows && !dbg.force_multilaunch;
  Plan p = p0;
  DeviceInfo di;
  RoundFn rfn = nullptr;
  int fit = 0;
  size_t smem = 0;
  if (narrow) {
    di = device_info();
    rfn = round_fn(p);
    // one streaming slice per remaining CU (at most kSlicesMax) plus the
    // selector block: every workgroup is resident at once
    int target = std::max(1, std::min(di.cus - 1, kRoundSlicesMax));
    if (dbg.round_slices > 0) target = std::min(target, dbg.round_slices);
    p.tiles_per_slice = (p.ntiles + target - 1) / target;
    p.G = (p.ntiles + p.tiles_per_slice - 1) / p.tiles_per_slice;
    // dynamic LDS: the frontier's head input, the keeper's top-N, then as
    // many resident W tiles as fit
    const int ncmax = nchunk_max(p);
    const size_t ubytes =
        ((size_t)p.rows_max * (p.r * (p.dtype ? 2 : 4) + 16) + 255) & ~(size_t)255;
    const size_t top = ubytes + (((size_t)p.R * p.N * (sizeof(uint64_t) + sizeof(int)) + 255) &
                                 ~(size_t)255);
    const size_t tile_bytes = (size_t)ncmax * 64 * 16;
    hipFuncAttributes attr{};
    int lds_max = 0;
    int dev = 0;
    if (di.cus >= 2 && hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
            hipSuccess &&
        hipFuncGetAttributes(&attr, (const void*)rfn) == hipSuccess) {
      const long room = (long)lds_max - (long)attr.sharedSizeBytes - (long)top - 1024;
      const int want =
          std::max(0, p.tiles_per_slice - resident_reg_tiles(ncmax, round_fold(p)) * kRoundWaves);
      const int cap = resident_lds_tiles_per_wave(ncmax) * kRoundWaves;
      p.lds_tiles = room > 0 ? (int)std::min<long>({room / (long)tile_bytes, (long)want, (long)cap})
                             : 0;
      p.lds_top_offset = (int)ubytes;
      p.lds_tile_offset = (int)top;
      smem = top + (size_t)p.lds_tiles * tile_bytes;
      if (hipFuncSetAttribute((const void*)rfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)smem) != hipSuccess ||
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&fit, (const void*)rfn, kRoundWaves * 64,
                                                       smem) != hipSuccess)
        fit = 0;
    }
  }
  p.tag = next_tag();
  if (narrow && fit > 0) {
    // a stage never legitimately waits 2 s; tests may shorten the bound so
    // that the waits give up (every workgroup still exits on its own)
    p.spin_ticks = dbg.wait_ticks >= 0 ? dbg.wait_ticks : 2 * di.ticks_per_s;
    // no word of an earlier use of the workspace may carry the call's tag
    {
      const int n = p.stages * p.rows_max * p.G * (p.kmax + kRecWords) + p.stages * p.rows_max;
      hipLaunchKernelGGL(clear_kernel, dim3(std::min((n + 255) / 256, 2048)), dim3(256), 0, st,
                         p);
    }
    void* args[] = {&p};
    const bool prof = profile_on();
    if (prof) profile_mark(st, "round_kernel");
    // An ordinary launch: the G + 1 workgroups (at most one per CU, checked
    // above) are all resident on an otherwise idle device.  A cooperative
    // launch would guarantee it even beside other work, but costs ~18 us of
    // dispatch per call here; with other kernels on the device a workgroup
    // may start late, which the bounded waits absorb (or the round aborts).
    const hipError_t e = hipLaunchKernel((const void*)rfn, dim3(p.G + 1),
                                         dim3(kRoundWaves * 64), args, smem, st);
    if (prof) profile_mark(st, "round_kernel");
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  p.unbounded = dbg.wide_unbounded;
  bool any_wide = false;
  for (int d = 0; d < p.B; ++d) any_wide = any_wide || stage_wide(p.mode, d, p.R, p.kk);
  if (any_wide && !p.unbounded)
    hipLaunchKernelGGL(probe_kernel, dim3(p.R * p.B), dim3(kProbeThreads), 0, st, p);
  hipLaunchKernelGGL(prologue_kernel, dim3(p.R), dim3(kSelectThreads), 0, st, p);
  const StageFn head = head_fn(p);
  const StageFn sel = select_fn(p.kmax);
  const StageFn head_thr = any_wide ? head_thr_fn(p) : nullptr;
  const StageFn mergesel = mergesel_fn(p.kmax);
  const int slices8 = (p.G + 7) / 8 * 8;
  for (int d = 0; d < p.B; ++d) {
    // head rows per request: the frontier, or the one shared row of the stage
    const int P = head_rows(p.mode, d, p.kk);
    const bool prof = profile_on();
    if (!stage_wide(p.mode, d, p.R, p.kk)) {
      // one column block: 4 waves split the slice's tiles; one WG per
      // request merges and selects
      if (prof) profile_mark(st, "head_kernel");
      hipLaunchKernelGGL(head, dim3(slices8), dim3(kHeadThreads), 0, st, p, d, P);
      if (prof) profile_mark(st, "head_kernel");
      hipLaunchKernelGGL(sel, dim3(p.R), dim3(kSelectThreads), 0, st, p, d, P);
    } else {
      // wide: up to 128 rows per workgroup, bounded candidates; one WG per
      // request merges its rows and selects
      const int cb = (p.R * P + kTile - 1) / kTile;
      const int ngrp = (cb + kWideWaves - 1) / kWideWaves;
      if (prof) profile_mark(st, "head_thr_kernel");
      hipLaunchKernelGGL(head_thr, dim3(slices8 * ngrp), dim3(kWideWaves * 64), 0, st, p, d, P);
      if (prof) profile_mark(st, "head_thr_kernel");
      hipLaunchKernelGGL(mergesel, dim3(p.R), dim3(kSelectThreads), 0, st, p, d, P);
    }
  }
  hipLaunchKernelGGL(emit_kernel, dim3(p.R), dim3(kEmitThreads), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_mask(const int* parent, const int* count, int R, int N, uint32_t* mask,
                       hipStream_t st) {
  hipLaunchKernelGGL(mask_kernel, dim3(R), dim3(kMaskThreads), 0, st, parent, count, N, mask);
  return hipGetLastError();
}

bool timeline_built() {
#ifdef PCTREE_TIMELINE
  return true;
#else
  return false;
#endif
}

hipError_t timeline_copy(long long* host, bool clear) {
#ifdef PCTREE_TIMELINE
  if (host) {
    const hipError_t e = hipMemcpyFromSymbol(host, HIP_SYMBOL(g_timeline), sizeof(g_timeline));
    if (e != hipSuccess) return e;
  }
  if (clear) {
    static const long long zero[kTimelineWho][kTimelineStages][kTimelineEvents] = {};
    return hipMemcpyToSymbol(HIP_SYMBOL(g_timeline), zero, sizeof(zero));
  }
  return hipSuccess;
#else
  (void)host;
  (void)clear;
  return hipErrorNotSupported;
#endif
}

}  // namespace pctree

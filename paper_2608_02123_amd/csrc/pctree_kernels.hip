// HIP kernels of the PCTree per-round tree builder for gfx950 (CDNA4).
//
// One round (Alg. 1) is enqueued as
//   prologue                       root node, frontier {x_t}, head input of x_t
//   for d in 0..B-1:
//     head_stream   (G x CB WGs)   Z = 1 L_d^T + U W for the frontier rows on
//                                  bf16/f32 MFMA, fused with an online row
//                                  logsumexp and per-row top-k; the V-wide
//                                  child logits never leave the chip (Eq. 2/3)
//     select        (R WGs)        merge the V-slices, score children (Eq. 4),
//                                  pick the next frontier (top-k of the layer)
//                                  and update the running global top-N
//   emit            (R WGs)        canonical emission + optional ancestor mask
//
// Ordering keys are unique 64-bit integers, so every selection is exact and
// deterministic:
//   child key  = ord(z)     << 32 | ~token                       (z desc, token asc)
//   node key   = ord(score) << 32 | (63-depth) << 26 | (2^20-1-token) << 6 | (63-slot)
//                                        (score desc, depth asc, token asc, slot asc)
// where ord() maps a float to an unsigned integer of the same order (-0 -> +0).
#include "pctree_plan.h"

#include <math.h>

#define PCTREE_EMIT_MAX_N 256
#define PCTREE_MASK_MAX_N 1024

namespace pctree {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -3.0e38f;  // "no value yet" for running maxima

__device__ __forceinline__ uint32_t f32_ord(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float f32_unord(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

__device__ __forceinline__ uint64_t child_key(float z, int tok) {
  return ((uint64_t)f32_ord(z) << 32) | (uint64_t)(~(uint32_t)tok);
}

__device__ __forceinline__ int child_key_token(uint64_t key) { return (int)(~(uint32_t)key); }

__device__ __forceinline__ float child_key_value(uint64_t key) {
  return f32_unord((uint32_t)(key >> 32));
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

template <int DT>
__device__ __forceinline__ float load_elem(const void* base, size_t i) {
  if (DT) return __uint_as_float((uint32_t)((const uint16_t*)base)[i] << 16);
  return ((const float*)base)[i];
}

// Write the head input of one frontier row: U[row][0..r) = act(E[tok], h_d).
__device__ void write_activation(const Plan& p, int row, int tok, const float* hd, int j0,
                                 int stride) {
  if (p.dtype) {
    uint16_t* u = (uint16_t*)p.U + (size_t)row * p.r;
    const uint16_t* e = (const uint16_t*)p.E + (size_t)tok * p.r;
    for (int j = j0; j < p.r; j += stride)
      u[j] = bf16_rne(silu_f32(__uint_as_float((uint32_t)e[j] << 16), hd[j]));
  } else {
    float* u = (float*)p.U + (size_t)row * p.r;
    const float* e = (const float*)p.E + (size_t)tok * p.r;
    for (int j = j0; j < p.r; j += stride) u[j] = silu_f32(e[j], hd[j]);
  }
}

// ---------------------------------------------------------------------------
// sorted (descending) fixed-length candidate lists held in registers
// ---------------------------------------------------------------------------
template <int K>
__device__ __forceinline__ void list_insert(uint64_t (&l)[K], uint64_t key) {
  l[K - 1] = key;
#pragma unroll
  for (int i = K - 1; i > 0; --i) {
    const uint64_t a = l[i - 1], b = l[i];
    const bool s = b > a;
    l[i - 1] = s ? b : a;
    l[i] = s ? a : b;
  }
}

// a <- top-K of (a u b); both sorted descending.  Elementwise max against the
// reversed b gives a bitonic sequence holding the top K; half-cleaners sort it.
template <int K>
__device__ __forceinline__ void list_merge(uint64_t (&a)[K], const uint64_t (&b)[K]) {
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const uint64_t x = a[i], y = b[K - 1 - i];
    a[i] = x > y ? x : y;
  }
#pragma unroll
  for (int j = K / 2; j > 0; j >>= 1) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if ((i & j) == 0) {
        const uint64_t x = a[i], y = a[i + j];
        const bool s = y > x;
        a[i] = s ? y : x;
        a[i + j] = s ? x : y;
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

// (m, s) pairs describe sum_i exp(z_i) = exp(m) * s; combine two of them.
__device__ __forceinline__ void lse_combine(float& m, float& s, float om, float os) {
  const float nm = fmaxf(m, om);
  s = s * exp2f((m - nm) * kLog2e) + os * exp2f((om - nm) * kLog2e);
  m = nm;
}

__device__ __forceinline__ void lse_combine_xor(float& m, float& s, int mask) {
  const float om = __shfl_xor(m, mask);
  const float os = __shfl_xor(s, mask);
  lse_combine(m, s, om, os);
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
__global__ __launch_bounds__(kEmitThreads) void prologue_kernel(Plan p) {
  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  int root = p.root[req];
  const bool bad = root < 0 || root >= p.V;
  if (bad) root = 0;
  if (tid == 0) {
    p.req_bad[req] = bad ? 1 : 0;
    const size_t nb = (size_t)req * p.maxpool;
    p.node_tok[nb] = root;
    p.node_par[nb] = -1;
    p.node_depth[nb] = 0;
    p.node_score[nb] = 0.0f;
    p.top_key[(size_t)req * p.N] = node_key(0.0f, 0, root, 0);
    p.top_node[(size_t)req * p.N] = 0;
    p.front_node[req * p.kk] = 0;
    p.front_tok[req * p.kk] = root;
    p.front_score[req * p.kk] = 0.0f;
  }
  if (p.t_token) {
    const int n = p.B * p.k;
    for (int i = tid; i < n; i += blockDim.x) {
      const size_t o = (size_t)req * n + i;
      const bool first = i == 0;
      p.t_token[o] = first ? root : -1;
      p.t_pslot[o] = -1;
      p.t_score[o] = first ? 0.0f : -INFINITY;
    }
  }
  write_activation(p, req * p.kk, root, p.h + (size_t)req * p.B * p.r, tid, blockDim.x);
}

// ---------------------------------------------------------------------------
// head stream: one WG per (V-slice, block of 16 frontier rows)
// ---------------------------------------------------------------------------
// MFMA 16x16xK with tokens as M and frontier rows as N: lane l feeds A row
// (token) l%16 and B column (row) l%16 with rank chunk group l/16, and
// receives C[token 4*(l/16)+i][row l%16], i = 0..3.
template <int DT, int NCMAX, int KMAX>
__global__ __launch_bounds__(kHeadThreads) void head_kernel(Plan p, int d, int P) {
  constexpr int KC = DT ? 32 : 16;  // rank elements per 16-byte chunk quad
  constexpr int ESZ = DT ? 2 : 4;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int rows = p.R * P;
  const int row = blockIdx.y * kTile + col;
  const bool row_ok = row < rows;
  const int req = row_ok ? row / P : 0;
  const int slot = row_ok ? row - req * P : 0;
  const int nc = p.nchunk;

  u32x4 bfrag[NCMAX];
  {
    const char* urow =
        (const char*)p.U + ((size_t)(req * p.kk + slot) * p.r + grp * (KC / 4)) * ESZ;
#pragma unroll
    for (int c = 0; c < NCMAX; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (c < nc && row_ok) v = *(const u32x4*)(urow + (size_t)c * KC * ESZ);
      bfrag[c] = v;
    }
  }
  const size_t lrow = ((size_t)req * p.B + d) * p.V;

  float m = kNegBig, s = 0.0f;
  uint64_t list[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) list[i] = 0;

  const int t0 = blockIdx.x * p.tiles_per_slice;
  const int t1 = min(t0 + p.tiles_per_slice, p.ntiles);
  for (int t = t0 + wave; t < t1; t += kHeadThreads / 64) {
    const int tokA = t * kTile + col;
    const char* wrow = (const char*)p.Wt + ((size_t)tokA * p.r + grp * (KC / 4)) * ESZ;
    u32x4 afrag[NCMAX];
#pragma unroll
    for (int c = 0; c < NCMAX; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (c < nc && tokA < p.V) v = *(const u32x4*)(wrow + (size_t)c * KC * ESZ);
      afrag[c] = v;
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCMAX; ++c)
      if (c < nc) acc = mfma_chunk<DT>(afrag[c], bfrag[c], acc);

    if (row_ok) {
      const int tb = t * kTile + grp * 4;
      float z[4];
      float tmax = kNegBig;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = tb + i;
        z[i] = tok < p.V ? acc[i] + load_elem<DT>(p.L, lrow + tok) : kNegBig;
        tmax = fmaxf(tmax, z[i]);
      }
      const float nm = fmaxf(m, tmax);
      float ss = s * exp2f((m - nm) * kLog2e);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (tb + i < p.V) ss += exp2f((z[i] - nm) * kLog2e);
      m = nm;
      s = ss;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (tb + i < p.V) {
          const uint64_t key = child_key(z[i], tb + i);
          if (key > list[KMAX - 1]) list_insert(list, key);
        }
      }
    }
  }

  // rows live in lanes col, col+16, col+32, col+48 of every wave
  list_merge_xor(list, 16);
  lse_combine_xor(m, s, 16);
  list_merge_xor(list, 32);
  lse_combine_xor(m, s, 32);

  __shared__ uint64_t sh_list[kHeadThreads / 64][kTile][KMAX];
  __shared__ float2 sh_ms[kHeadThreads / 64][kTile];
  if (grp == 0) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) sh_list[wave][col][i] = list[i];
    sh_ms[wave][col] = make_float2(m, s);
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) list[i] = sh_list[grp][col][i];
    m = sh_ms[grp][col].x;
    s = sh_ms[grp][col].y;
    list_merge_xor(list, 16);
    lse_combine_xor(m, s, 16);
    list_merge_xor(list, 32);
    lse_combine_xor(m, s, 32);
    if (grp == 0 && row_ok) {
      const size_t o = (size_t)blockIdx.x * p.rows_max + row;
      uint64_t* dst = p.part_key + o * KMAX;
#pragma unroll
      for (int i = 0; i < KMAX; ++i) dst[i] = list[i];
      p.part_ms[o] = make_float2(m, s);
    }
  }
}

// ---------------------------------------------------------------------------
// select: one WG per request after every head launch
// ---------------------------------------------------------------------------
template <int KMAX>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(Plan p, int d, int P) {
  constexpr int NW = kSelectThreads / 64;
  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int kk = p.kk;
  const int ncand = P * kk;

  __shared__ uint64_t sh_wlist[NW][KMAX];
  __shared__ float2 sh_wms[NW];
  __shared__ uint64_t sh_rowkeys[16][KMAX];
  __shared__ float sh_lse[16];
  __shared__ uint64_t sh_ckey[256];
  __shared__ int sh_rank[256];
  __shared__ uint64_t sh_tkey[256];

  // 1. merge the G slice lists of every frontier row of this request
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
      const size_t o = (size_t)g * p.rows_max + grow;
      uint64_t other[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) other[i] = p.part_key[o * KMAX + i];
      list_merge(list, other);
      const float2 ms = p.part_ms[o];
      lse_combine(m, s, ms.x, ms.y);
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
    // lanes 0..wpr-1 of the row's first wave combine the row's waves
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
      for (int i = 0; i < KMAX; ++i) sh_rowkeys[prow][i] = list[i];
      sh_lse[prow] = m + logf(s);
    }
  }
  __syncthreads();

  // 2. children of every frontier row, scored (Eq. 4), into the pool
  const int nbase = d == 0 ? 1 : 1 + kk + (d - 1) * kk * kk;  // pool id of the first candidate
  const size_t pb = (size_t)req * p.maxpool;
  if (tid < ncand) {
    const int pr = tid / kk;
    const int j = tid - pr * kk;
    const uint64_t ck = sh_rowkeys[pr][j];
    // every row holds >= k' real keys (V >= k'); the clamp only keeps a
    // corrupted key from indexing E out of bounds
    const int tok = min(max(child_key_token(ck), 0), p.V - 1);
    const float lp = child_key_value(ck) - sh_lse[pr];
    const float score = p.front_score[req * kk + pr] + lp;
    const int id = nbase + tid;
    p.node_tok[pb + id] = tok;
    p.node_par[pb + id] = p.front_node[req * kk + pr];
    p.node_depth[pb + id] = d + 1;
    p.node_score[pb + id] = score;
    sh_ckey[tid] = node_key(score, d + 1, tok, pr);
  }
  const int cur = d & 1;
  const int ncur = min(p.N, nbase);
  const uint64_t* tk = p.top_key + ((size_t)cur * p.R + req) * p.N;
  const int* tn = p.top_node + ((size_t)cur * p.R + req) * p.N;
  if (tid >= 256 && tid < 256 + ncur) sh_tkey[tid - 256] = tk[tid - 256];
  __syncthreads();

  // 3. rank of every candidate within the layer (the layer order)
  if (tid < ncand) {
    const uint64_t key = sh_ckey[tid];
    int rank = 0;
    for (int c = 0; c < ncand; ++c) rank += sh_ckey[c] > key;
    sh_rank[tid] = rank;
  }
  __syncthreads();

  // 4. next frontier = the k' best candidates of the layer
  const bool more = d + 1 < p.B;
  if (more && tid < ncand && sh_rank[tid] < kk) {
    const int slot = sh_rank[tid];
    const int pr = tid / kk;
    const int id = nbase + tid;
    const int tok = p.node_tok[pb + id];
    const float score = p.node_score[pb + id];
    p.front_node[req * kk + slot] = id;
    p.front_tok[req * kk + slot] = tok;
    p.front_score[req * kk + slot] = score;
    if (p.t_token) {
      const size_t o = ((size_t)req * p.B + d + 1) * p.k + slot;
      p.t_token[o] = tok;
      p.t_pslot[o] = pr;
      p.t_score[o] = score;
    }
  }

  // 5. running global top-N: merge the sorted list with the ranked layer
  const int nxt = cur ^ 1;
  uint64_t* ok = p.top_key + ((size_t)nxt * p.R + req) * p.N;
  int* on = p.top_node + ((size_t)nxt * p.R + req) * p.N;
  if (tid < ncand) {
    const uint64_t key = sh_ckey[tid];
    int pos = sh_rank[tid];
    for (int i = 0; i < ncur; ++i) pos += sh_tkey[i] > key;
    if (pos < p.N) {
      ok[pos] = key;
      on[pos] = nbase + tid;
    }
  } else if (tid >= 256 && tid < 256 + ncur) {
    const int i = tid - 256;
    const uint64_t key = sh_tkey[i];
    int pos = i;
    for (int c = 0; c < ncand; ++c) pos += sh_ckey[c] > key;
    if (pos < p.N) {
      ok[pos] = key;
      on[pos] = tn[i];
    }
  }
  __syncthreads();

  // 6. head input of the next frontier
  if (more) {
    const float* hd = p.h + ((size_t)req * p.B + d + 1) * p.r;
    const int n = kk * p.r;
    for (int e = tid; e < n; e += kSelectThreads) {
      const int slot = e / p.r;
      const int j = e - slot * p.r;
      const int tok = p.front_tok[req * kk + slot];
      // one element at a time: write_activation() with a stride over j
      if (p.dtype) {
        const uint16_t* er = (const uint16_t*)p.E + (size_t)tok * p.r;
        ((uint16_t*)p.U)[(size_t)(req * kk + slot) * p.r + j] =
            bf16_rne(silu_f32(__uint_as_float((uint32_t)er[j] << 16), hd[j]));
      } else {
        const float* er = (const float*)p.E + (size_t)tok * p.r;
        ((float*)p.U)[(size_t)(req * kk + slot) * p.r + j] = silu_f32(er[j], hd[j]);
      }
    }
  }
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
// Level by level, every node of the level ranks itself among its level.
__global__ __launch_bounds__(kEmitThreads) void emit_kernel(Plan p) {
  __shared__ int sh_node[kEmitThreads], sh_emit[kEmitThreads], sh_par_emit[kEmitThreads];
  __shared__ uint64_t sh_skey[kEmitThreads];
  __shared__ int lev_cnt[64], lev_off[65], lev_fill[64], lev_mem[kEmitThreads];
  __shared__ uint32_t sh_words[kEmitThreads * (PCTREE_EMIT_MAX_N / 32)];

  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  const int kk = p.kk;
  const int pool = 1 + kk + (p.B - 1) * kk * kk;
  int count = min(p.N, pool);
  if (p.req_bad[req]) count = 0;
  const int fin = p.B & 1;
  const size_t pb = (size_t)req * p.maxpool;

  if (tid < 64) {
    lev_cnt[tid] = 0;
    lev_fill[tid] = 0;
  }
  __syncthreads();
  int node = -1, dep = -1, tok = -1, pnode = -1;
  float score = 0.0f;
  if (tid < count) {
    node = p.top_node[((size_t)fin * p.R + req) * p.N + tid];
    dep = p.node_depth[pb + node];
    tok = p.node_tok[pb + node];
    pnode = p.node_par[pb + node];
    score = p.node_score[pb + node];
    sh_node[tid] = node;
    atomicAdd(&lev_cnt[dep], 1);
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
  __syncthreads();
  if (tid < count) lev_mem[lev_off[dep] + atomicAdd(&lev_fill[dep], 1)] = tid;
  __syncthreads();

  int emit = -1, pemit = -1;
  for (int l = 0; l <= p.B; ++l) {
    if (dep == l) {
      if (l > 0) {
        for (int q = lev_off[l - 1]; q < lev_off[l]; ++q) {
          const int j = lev_mem[q];
          if (sh_node[j] == pnode) pemit = sh_emit[j];
        }
      }
      sh_skey[tid] = ((uint64_t)(uint32_t)(pemit + 1) << 32) | (uint32_t)tok;
    }
    __syncthreads();
    if (dep == l) {
      const uint64_t key = sh_skey[tid];
      int rank = 0;
      for (int q = lev_off[l]; q < lev_off[l + 1]; ++q) rank += sh_skey[lev_mem[q]] < key;
      emit = lev_off[l] + rank;
      sh_emit[tid] = emit;
    }
    __syncthreads();
  }

  const size_t ob = (size_t)req * p.N;
  if (tid < count) {
    p.o_token[ob + emit] = tok;
    p.o_parent[ob + emit] = pemit;
    p.o_depth[ob + emit] = dep;
    p.o_position[ob + emit] = p.prefix[req] + dep;
    p.o_logprob[ob + emit] = score;
    sh_par_emit[emit] = pemit;
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
    __syncthreads();
    mask_rows(sh_par_emit, count, p.N, p.o_mask + (size_t)req * p.N * ((p.N + 31) / 32),
              sh_words, PCTREE_EMIT_MAX_N / 32);
  }
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
typedef void (*HeadFn)(Plan, int, int);
typedef void (*SelectFn)(Plan, int, int);

template <int DT, int NCMAX>
HeadFn head_for_kmax(int kmax) {
  switch (kmax) {
    case 1: return head_kernel<DT, NCMAX, 1>;
    case 2: return head_kernel<DT, NCMAX, 2>;
    case 4: return head_kernel<DT, NCMAX, 4>;
    case 8: return head_kernel<DT, NCMAX, 8>;
    default: return head_kernel<DT, NCMAX, 16>;
  }
}

HeadFn head_fn(const Plan& p) {
  if (p.dtype) {
    if (p.nchunk <= 4) return head_for_kmax<1, 4>(p.kmax);
    if (p.nchunk <= 8) return head_for_kmax<1, 8>(p.kmax);
    return head_for_kmax<1, 16>(p.kmax);
  }
  if (p.nchunk <= 2) return head_for_kmax<0, 2>(p.kmax);
  return head_for_kmax<0, 8>(p.kmax);
}

SelectFn select_fn(int kmax) {
  switch (kmax) {
    case 1: return select_kernel<1>;
    case 2: return select_kernel<2>;
    case 4: return select_kernel<4>;
    case 8: return select_kernel<8>;
    default: return select_kernel<16>;
  }
}

}  // namespace

hipError_t launch_round(const Plan& p, hipStream_t st) {
  hipLaunchKernelGGL(prologue_kernel, dim3(p.R), dim3(kEmitThreads), 0, st, p);
  const HeadFn head = head_fn(p);
  const SelectFn sel = select_fn(p.kmax);
  for (int d = 0; d < p.B; ++d) {
    const int P = d == 0 ? 1 : p.kk;
    const int cb = (p.R * P + kTile - 1) / kTile;
    const bool prof = profile_on();
    if (prof) profile_mark(st);
    hipLaunchKernelGGL(head, dim3(p.G, cb), dim3(kHeadThreads), 0, st, p, d, P);
    if (prof) profile_mark(st);
    hipLaunchKernelGGL(sel, dim3(p.R), dim3(kSelectThreads), 0, st, p, d, P);
  }
  hipLaunchKernelGGL(emit_kernel, dim3(p.R), dim3(kEmitThreads), 0, st, p);
  return hipGetLastError();
}

const char* dominant_kernel_name() { return "head_kernel"; }

hipError_t launch_mask(const int* parent, const int* count, int R, int N, uint32_t* mask,
                       hipStream_t st) {
  hipLaunchKernelGGL(mask_kernel, dim3(R), dim3(kMaskThreads), 0, st, parent, count, N, mask);
  return hipGetLastError();
}

}  // namespace pctree

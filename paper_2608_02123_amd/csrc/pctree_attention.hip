// Tree-masked verification attention of one target layer (paper Sec. 4.2
// and App. A, "Tensor implementation"): the emitted tree is checked in one
// target forward, in which tree node i may attend to the verified prefix, to
// itself and to its ancestors.  Cache slot prefix_len + j holds tree node j,
// so the admitted slots of node i are [0, prefix_len) and prefix_len + j for
// every set bit j < count of its ancestor-mask row.
//
// Layout (bf16): q [R][N][Hq][D], k and v [R][Hkv][C][D], out [R][N][Hq][D];
// query head h reads key/value head h / g, g = Hq / Hkv.
//
// One workgroup (4 waves of 32 rows) takes 128 query rows of one key/value
// head, row rho = node * g + (h mod g), and a run of key slots (the whole
// admitted range, or one split of it when there are too few workgroups to
// fill the chip).  Key slots go through LDS 64 at a time (register-prefetched
// one chunk ahead): K row-major, V transposed, shared by the four waves, with
// a 64-bit window per tree node of which of the chunk's slots it admits.
// Each wave owns two 16-row column tiles and computes, on bf16 MFMA 16x16x32
// with fp32 accumulation (every K and V fragment read from LDS serves both
// tiles),
//   S^T = K Q^T   (a 32-key x 16-row tile pair, contraction over D), then
//   O^T += V^T P^T (D x 16 rows, contraction over the 32 keys),
// with an online softmax in base 2 (one update per chunk).  The two K tiles of a pair take keys
// {8c..8c+3} and {8c+4..8c+7} on row group c, so that every lane ends up with
// the scores of 8 consecutive keys of its query row: exactly the B operand
// of the second product, with no data movement between lanes.  Split runs
// leave (max, sum, unnormalised output) per row in the workspace and a
// second kernel merges them.
#include "pctree.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pctree_attention.h"

namespace pctree {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;      // 4 waves
constexpr int kColTiles = 2;       // 16-row MFMA column tiles per wave
constexpr int kRowsPerWave = 16 * kColTiles;
constexpr int kRowsPerBlock = 4 * kRowsPerWave;  // query rows of one workgroup
constexpr int kChunk = 64;         // key slots per LDS stage (two 32-slot halves)
constexpr int kKPad = 8;           // bf16 padding of an LDS K row
constexpr int kVPad = 8;           // bf16 padding of an LDS V^T row
constexpr int kMaxSplits = 32;     // slot runs merged by one merge thread
constexpr int kXcds = 8;           // L2 domains the dispatcher deals workgroups over
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 8;     // slot runs whose loads one merge thread issues together
constexpr float kNegInf = -__builtin_inff();

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Two floats to packed bf16 (round to nearest even), the low half first.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// 16-byte group of K row `row` that holds d group `dg` in LDS.  Rows are
// D + 8 bf16 long (a shift of 4 banks per row), and the fragment reads of a
// 16-lane group touch rows {0..3, 8..11, 16..19, 24..27} (+ 4, + 32): rows 16
// apart would share banks, so rows with bit 4 set swap d groups 4 apart.
__device__ __forceinline__ int kswz(int row, int dg) { return dg ^ (((row >> 4) & 1) << 2); }

// Low `n` bits set, n in [0, 64].
__device__ __forceinline__ uint64_t low_bits(int n) {
  return n >= 64 ? ~0ull : ((1ull << n) - 1ull);
}

// Admitted key range of request r: [0, prefix + count) clamped to the cache.
struct ReqRange {
  int prefix, cnt, end;
};

__device__ __forceinline__ ReqRange req_range(const AttnArgs& a, int r) {
  ReqRange q;
  q.cnt = min(max(a.count[r], 0), a.N);
  q.prefix = min(max(a.prefix_len[r], 0), a.C);
  q.end = min(q.prefix + q.cnt, a.C);
  return q;
}

// Workgroups are dealt round-robin over the XCDs, each with its own L2.  The
// query blocks of one (request, kv head, slot run) read the same K and V, so
// they are given block ids that land on one XCD: block b serves group
// (b / 8 / qblocks) * 8 + b % 8, query block (b / 8) % qblocks.  Ids past the
// last group return at once.
struct Work {
  int r, kvh, split, qb;
  bool ok;
};

__device__ __forceinline__ Work work_of(const AttnArgs& a) {
  const int b = blockIdx.x;
  const int j = b / kXcds;
  const int grp = (j / a.qblocks) * kXcds + b % kXcds;
  Work w;
  w.ok = grp < a.R * a.Hkv * a.nsplit;
  w.qb = j % a.qblocks;
  w.split = grp % a.nsplit;
  w.kvh = grp / a.nsplit % a.Hkv;
  w.r = grp / a.nsplit / a.Hkv;
  return w;
}

// Maximum over the four lanes that hold one query row (lanes l, l ^ 16,
// l ^ 32, l ^ 48), exchanged on the VALU (v_permlane{16,32}_swap return the
// lane's own value and its partner's, in a lane-dependent order that a
// maximum does not care about).
__device__ __forceinline__ float row_max4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                   false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                   false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Online softmax of one 16-row column tile over a 64-slot chunk.  s[h][t]
// holds the raw scores q.k of half h, tile t (slots 32 h + 8 grp + 4 t + e);
// `adm` has bit 8 h + i set when slot 32 h + 8 grp + i is admitted (ignored
// when `all`).  The running maximum m is kept in raw units, which needs
// scale > 0: the weights are 2^(scale log2(e) (s - m)).  Writes the weights
// as bf16 B operands bp[h] and returns the factor the accumulated output must
// be scaled by.
__device__ __forceinline__ float softmax_chunk(const f32x4 (&s)[2][2], uint32_t adm, bool all,
                                               float c, float& m, float& l, u32x4 (&bp)[2]) {
  float v[16];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[8 * h + e] = s[h][0][e];
      v[8 * h + 4 + e] = s[h][1][e];
    }
  if (!all) {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = ((adm >> i) & 1u) ? v[i] : kNegInf;
  }
  float cmax = v[0];
#pragma unroll
  for (int i = 1; i < 16; ++i) cmax = fmaxf(cmax, v[i]);
  const float mn = fmaxf(m, row_max4(cmax));
  const float alpha = mn == m ? 1.0f : exp2_hw((m - mn) * c);  // m = -inf: 0
  const float off = mn == kNegInf ? 0.0f : mn * c;  // nothing admitted yet: every weight 0
  float ps = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    v[i] = exp2_hw(__builtin_fmaf(v[i], c, -off));
    ps += v[i];
  }
  m = mn;
  l = l * alpha + ps;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < 4; ++i) bp[h][i] = pack_bf16(v[8 * h + 2 * i], v[8 * h + 2 * i + 1]);
  return alpha;
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_kernel(AttnArgs a) {
  constexpr int KS = D / 32;  // contraction steps of S = K Q^T
  constexpr int DT = D / 16;  // 16-wide d tiles of O
  constexpr int KROW = D + kKPad;
  constexpr int VROW = kChunk + kVPad;
  constexpr int DG = D / 8;   // 16-byte groups of a row
  constexpr int CT = kColTiles;
  __shared__ __attribute__((aligned(16))) uint16_t sK[kChunk * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * VROW];
  __shared__ uint64_t sWin[kRowsPerBlock];  // admitted slots of the chunk, per node

  const Work wk = work_of(a);
  if (!wk.ok) return;
  const int r = wk.r, kvh = wk.kvh, split = wk.split;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;

  // this lane's query rows (MFMA column col of each tile): rho = node * g + (h mod g)
  const int rows_kv = a.N * a.g;
  const int n0 = wk.qb * kRowsPerBlock / a.g;  // first node of the block
  const int nn = min((wk.qb * kRowsPerBlock + kRowsPerBlock - 1) / a.g - n0 + 1, a.N - n0);
  bool row_in[CT];
  int node[CT], hq[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int rho = wk.qb * kRowsPerBlock + wave * kRowsPerWave + 16 * c + col;
    row_in[c] = rho < rows_kv;
    node[c] = row_in[c] ? rho / a.g : 0;
    hq[c] = kvh * a.g + (row_in[c] ? rho % a.g : 0);
  }

  // Q^T fragments (8 consecutive d of the row per contraction step), issued
  // before the request's lengths are known
  u32x4 bq[CT][KS];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const uint16_t* qrow = a.q + (((size_t)r * a.N + node[c]) * a.Hq + hq[c]) * D + grp * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) bq[c][s] = *(const u32x4*)(qrow + s * 32);
  }

  // Staging maps.  K: thread -> d group st_dg of key rows st_row + 16 i.
  // V: thread -> key pair (2 vp, 2 vp + 1) and d groups vdg + 8 j, so that
  // the 64 lanes of a wave write 64 different LDS banks of the transposed
  // tile (lane pairs 32 apart sit 8 d rows apart: 288 bytes, 8 banks + 32).
  const int st_dg = tid & 15, st_row = tid >> 4;
  const bool st_on = st_dg < DG;
  const int vp = tid & 31, vdg = tid >> 5;
  constexpr int VJ = DG / 8;  // V d groups per thread (1 or 2)
  const size_t kvbase = ((size_t)r * a.Hkv + kvh) * a.C;
  const uint16_t* kbase_p = a.k + kvbase * D + st_dg * 8;
  const uint16_t* vbase_p = a.v + kvbase * D + vdg * 8;
  u32x4 nk[4], nv[2 * VJ];
  // raw loads of chunk c0 (slot addresses clamped into the cache; slots past
  // the run are zeroed when staged)
  auto fetch = [&](int c0) {
    if (st_on) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        nk[i] = *(const u32x4*)(kbase_p + (size_t)min(c0 + st_row + 16 * i, a.C - 1) * D);
    }
    const size_t s0 = (size_t)min(c0 + 2 * vp, a.C - 1) * D;
    const size_t s1 = (size_t)min(c0 + 2 * vp + 1, a.C - 1) * D;
#pragma unroll
    for (int j = 0; j < VJ; ++j) {
      nv[2 * j] = *(const u32x4*)(vbase_p + s0 + 64 * j);
      nv[2 * j + 1] = *(const u32x4*)(vbase_p + s1 + 64 * j);
    }
  };
  const int kbeg = split * a.split_keys;
  fetch(kbeg);  // kbeg < C by construction of the runs

  const ReqRange rr = req_range(a, r);
  const int kend = min(kbeg + a.split_keys, rr.end);
  if (a.nsplit > 1 && kbeg >= rr.end) return;  // empty run: the merge skips it
  bool row_live[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    row_live[c] = row_in[c] && node[c] < rr.cnt;
    if (!row_live[c]) {
#pragma unroll
      for (int s = 0; s < KS; ++s) bq[c][s] = u32x4{0u, 0u, 0u, 0u};
    }
  }

  // Admission windows: thread t < nn keeps, for node n0 + t, the three mask
  // words that cover the chunk's tree slots (bit j of the mask row is tree
  // node j, at slot prefix + j).
  const uint32_t* mrow_g = a.mask + ((size_t)r * a.N + n0 + min(tid, nn - 1)) * a.NW;
  uint32_t mw0 = 0, mw1 = 0, mw2 = 0;
  auto fetch_mask = [&](int c0) {
    mw0 = mw1 = mw2 = 0;
    if (tid >= nn || c0 + kChunk <= rr.prefix || c0 >= kend) return;  // no tree slot
    const int j0 = c0 - rr.prefix;
    const int wb = j0 >= 0 ? j0 >> 5 : -((31 - j0) >> 5);  // floor(j0 / 32)
    if (wb >= 0 && wb < a.NW) mw0 = mrow_g[wb];
    if (wb + 1 >= 0 && wb + 1 < a.NW) mw1 = mrow_g[wb + 1];
    if (wb + 2 >= 0 && wb + 2 < a.NW) mw2 = mrow_g[wb + 2];
  };
  fetch_mask(kbeg);

  f32x4 o[CT][DT];
  float m[CT], l[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    m[c] = kNegInf;
    l[c] = 0.0f;
#pragma unroll
    for (int t = 0; t < DT; ++t) o[c][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto stage = [&](int c0) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    if (st_on) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = st_row + 16 * i;
        *(u32x4*)(sK + row * KROW + kswz(row, st_dg) * 8) = c0 + row < kend ? nk[i] : z;
      }
    }
    const bool lo_ok = c0 + 2 * vp < kend, hi_ok = c0 + 2 * vp + 1 < kend;
#pragma unroll
    for (int j = 0; j < VJ; ++j) {
      const u32x4 lo = lo_ok ? nv[2 * j] : z;
      const u32x4 hi = hi_ok ? nv[2 * j + 1] : z;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // d = 8 (vdg + 8 j) + 2e (low halves) and + 1 (high halves); keys 2 vp, + 1
        uint16_t* dst = sV + ((vdg + 8 * j) * 8 + 2 * e) * VROW + 2 * vp;
        *(uint32_t*)dst = (lo[e] & 0xffffu) | (hi[e] << 16);
        *(uint32_t*)(dst + VROW) = (lo[e] >> 16) | (hi[e] & 0xffff0000u);
      }
    }
    if (tid < nn) {
      // bit i: slot c0 + i is admitted for node n0 + tid
      uint64_t win = 0;
      if (n0 + tid < rr.cnt) {
        const int j0 = c0 - rr.prefix;
        const int sh = j0 & 31;  // j0 - 32 floor(j0 / 32)
        const uint64_t lo64 = ((uint64_t)mw1 << 32) | mw0;
        const uint64_t tree = sh ? (lo64 >> sh) | ((uint64_t)mw2 << (64 - sh)) : lo64;
        const int np = min(max(rr.prefix - c0, 0), kChunk);
        win = (low_bits(np) | (tree & ~low_bits(np))) & low_bits(min(max(kend - c0, 0), kChunk));
      }
      sWin[tid] = win;
    }
  };

  // A-operand rows of an S^T tile pair: tile 0 holds keys 8c + e, tile 1 keys
  // 8c + 4 + e, for MFMA row 4c + e (c = col / 4, e = col % 4)
  const int krow0 = 8 * (col >> 2) + (col & 3);

  for (int c0 = kbeg; c0 < kend; c0 += kChunk) {
    __syncthreads();  // the previous chunk is no longer read
    stage(c0);
    __syncthreads();
    if (c0 + kChunk < kend) {
      fetch(c0 + kChunk);
      fetch_mask(c0 + kChunk);
    }
    uint64_t win[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) win[c] = row_live[c] ? sWin[node[c] - n0] : 0ull;
    // every slot of the chunk admitted for every live row: no masking (rows
    // past the tree then take weights like the rest and are written as zeros)
    const bool full = c0 + kChunk <= min(kend, rr.prefix);

    // S^T for both halves and both column tiles: 8 independent chains
    f32x4 sacc[CT][2][2];
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) sacc[c][h][0] = sacc[c][h][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < KS; ++k) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row0 = 32 * h + krow0;
        const u32x4 a0 = *(const u32x4*)(sK + row0 * KROW + kswz(row0, 4 * k + grp) * 8);
        const u32x4 a1 =
            *(const u32x4*)(sK + (row0 + 4) * KROW + kswz(row0 + 4, 4 * k + grp) * 8);
#pragma unroll
        for (int c = 0; c < CT; ++c) {
          sacc[c][h][0] = mfma_bf16(a0, bq[c][k], sacc[c][h][0]);
          sacc[c][h][1] = mfma_bf16(a1, bq[c][k], sacc[c][h][1]);
        }
      }
    }
    u32x4 bp[CT][2];
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const uint32_t adm = (uint32_t)(win[c] >> (8 * grp)) & 0xffu |
                           ((uint32_t)(win[c] >> (32 + 8 * grp)) & 0xffu) << 8;
      const float alpha =
          softmax_chunk(sacc[c], adm, full, a.scale_log2, m[c], l[c], bp[c]);
      if (__any(alpha != 1.0f)) {  // rescale only when some row raised its max
#pragma unroll
        for (int t = 0; t < DT; ++t) o[c][t] *= alpha;
      }
    }
    const uint16_t* va = sV + col * VROW + 8 * grp;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const u32x4 av0 = *(const u32x4*)(va + t * 16 * VROW);
      const u32x4 av1 = *(const u32x4*)(va + t * 16 * VROW + 32);
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        o[c][t] = mfma_bf16(av0, bp[c][0], o[c][t]);
        o[c][t] = mfma_bf16(av1, bp[c][1], o[c][t]);
      }
    }
  }

#pragma unroll
  for (int c = 0; c < CT; ++c) {
    // the row's sum over its four lane groups
    float lc = l[c];
    lc += __shfl_xor(lc, 16, 64);
    lc += __shfl_xor(lc, 32, 64);
    if (!row_in[c]) continue;
    const size_t qidx = ((size_t)r * a.N + node[c]) * a.Hq + hq[c];  // (request, node, head)
    if (a.nsplit == 1) {
      const float inv = row_live[c] && lc > 0.0f ? 1.0f / lc : 0.0f;
      uint16_t* orow = a.out + qidx * D;
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const f32x4 v = o[c][t] * inv;
        u32x2 w;
        w[0] = pack_bf16(v[0], v[1]);
        w[1] = pack_bf16(v[2], v[3]);
        *(u32x2*)(orow + t * 16 + 4 * grp) = w;
      }
    } else {
      const size_t prow = (size_t)split * a.R * a.N * a.Hq + qidx;
      float* po = a.part_o + prow * D;
#pragma unroll
      for (int t = 0; t < DT; ++t) *(f32x4*)(po + t * 16 + 4 * grp) = o[c][t];
      if (grp == 0) {
        a.part_ml[2 * prow] = row_live[c] ? m[c] : kNegInf;
        a.part_ml[2 * prow + 1] = row_live[c] ? lc : 0.0f;
      }
    }
  }
}

// Merge of the slot runs: D / 4 threads per row of (request, node, head), 4
// consecutive d each.  Only the runs that hold admitted slots were written.
// The runs are read in batches of kMergeBatch whose loads are all issued
// before any is used (clamped to a written run), folded into a running
// (max, sum, output) per batch.
template <int D>
__global__ __launch_bounds__(kMergeThreads) void attn_merge_kernel(AttnArgs a) {
  constexpr int TPR = D / 4;                // threads per row
  constexpr int RPB = kMergeThreads / TPR;  // rows per workgroup
  const size_t rows = (size_t)a.R * a.N * a.Hq;
  const size_t qidx = (size_t)blockIdx.x * RPB + threadIdx.x / TPR;
  const int d = (threadIdx.x % TPR) * 4;
  if (qidx >= rows) return;
  const int r = (int)(qidx / ((size_t)a.N * a.Hq));
  const int node = (int)(qidx / a.Hq % a.N);
  const ReqRange rr = req_range(a, r);
  const int ns = node < rr.cnt ? min(a.nsplit, (rr.end + a.split_keys - 1) / a.split_keys) : 0;
  float M = kNegInf, L = 0.0f;
  f32x4 O = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < ns; s0 += kMergeBatch) {
    float ms[kMergeBatch], ls[kMergeBatch];
    f32x4 os[kMergeBatch];
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const size_t prow = (size_t)min(s0 + i, ns - 1) * rows + qidx;
      ms[i] = a.part_ml[2 * prow];
      ls[i] = a.part_ml[2 * prow + 1];
      os[i] = *(const f32x4*)(a.part_o + prow * D + d);
    }
    float bm = kNegInf;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i)
      if (s0 + i < ns) bm = fmaxf(bm, ms[i]);
    const float Mn = fmaxf(M, bm);
    if (Mn == kNegInf) continue;  // no admitted slot so far
    const float sc = M == kNegInf ? 0.0f : exp2_hw((M - Mn) * a.scale_log2);
    L *= sc;
    O *= sc;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      // a run with no admitted slot of this row (max -inf) adds nothing
      if (s0 + i < ns && ms[i] != kNegInf) {
        const float w = exp2_hw((ms[i] - Mn) * a.scale_log2);  // maxima in raw units
        L += w * ls[i];
        O += os[i] * w;
      }
    }
    M = Mn;
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  u32x2 w;
  w[0] = pack_bf16(O[0] * inv, O[1] * inv);
  w[1] = pack_bf16(O[2] * inv, O[3] * inv);
  *(u32x2*)(a.out + qidx * D + d) = w;
}

}  // namespace

AttnPlan plan_attention(int R, int N, int Hq, int Hkv, int D, int C, int cus) {
  AttnPlan p;
  const int g = Hq / Hkv;
  p.qblocks = (N * g + kRowsPerBlock - 1) / kRowsPerBlock;
  const long long base = (long long)R * Hkv * p.qblocks;
  const int chunks = (C + kChunk - 1) / kChunk;
  // enough workgroups for one per two compute units (more runs cost more in
  // the merge pass than they save here)
  int ns = 1;
  const int target = cus / 2;
  if (base < target) ns = (int)((target + base - 1) / base);
  ns = ns < chunks ? ns : chunks;
  ns = ns < kMaxSplits ? ns : kMaxSplits;
  ns = ns < 1 ? 1 : ns;
  const int per = (chunks + ns - 1) / ns;  // chunks per run
  p.split_keys = per * kChunk;
  p.nsplit = (chunks + per - 1) / per;
  const long long groups = (long long)R * Hkv * p.nsplit;
  p.blocks = (int)(((groups + kXcds - 1) / kXcds) * kXcds * p.qblocks);
  const size_t rows = (size_t)R * N * Hq;
  p.ws_bytes = p.nsplit > 1 ? (size_t)p.nsplit * rows * (D + 2) * sizeof(float) + 256 : 0;
  return p;
}

hipError_t launch_attention(AttnArgs a, int blocks, int D, hipStream_t stream) {
  if (D == 128)
    attn_kernel<128><<<blocks, kThreads, 0, stream>>>(a);
  else
    attn_kernel<64><<<blocks, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  const size_t rows = (size_t)a.R * a.N * a.Hq;
  const int rpb = kMergeThreads / (D / 4);
  const unsigned mblocks = (unsigned)((rows + rpb - 1) / rpb);
  if (D == 128)
    attn_merge_kernel<128><<<mblocks, kMergeThreads, 0, stream>>>(a);
  else
    attn_merge_kernel<64><<<mblocks, kMergeThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace pctree

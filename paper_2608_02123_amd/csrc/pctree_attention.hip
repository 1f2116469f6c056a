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
// One workgroup (4 waves) takes 64 query rows of one key/value head, row
// rho = node * g + (h mod g), and a run of key slots (the whole admitted range,
// or one split of it when there are too few workgroups to fill the chip).
// Key slots go through LDS 32 at a time: K row-major, V transposed, shared by
// the four waves.  Each wave owns 16 query rows and computes, on bf16 MFMA
// 16x16x32 with fp32 accumulation,
//   S^T = K Q^T   (a 32-key x 16-row tile pair, contraction over D), then
//   O^T += V^T P^T (D x 16 rows, contraction over the 32 keys),
// with an online softmax in base 2.  The two K tiles of a pair take keys
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
constexpr int kRowsPerWave = 16;   // query rows of one wave (MFMA columns)
constexpr int kRowsPerBlock = 64;  // query rows of one workgroup
constexpr int kChunk = 32;         // key slots per LDS stage
constexpr int kKPad = 8;           // bf16 padding of an LDS K row
constexpr int kVPad = 8;           // bf16 padding of an LDS V^T row
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7fffu + ((b >> 16) & 1u);
  return b >> 16;
}

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

template <int D>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnArgs a) {
  constexpr int KS = D / 32;  // contraction steps of S = K Q^T
  constexpr int DT = D / 16;  // 16-wide d tiles of O
  constexpr int KROW = D + kKPad;
  constexpr int VROW = kChunk + kVPad;
  __shared__ __attribute__((aligned(16))) uint16_t sK[kChunk * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * VROW];

  const int qb = blockIdx.x % a.qblocks;
  const int split = blockIdx.x / a.qblocks;
  const int kvh = blockIdx.y;
  const int r = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;

  const ReqRange rr = req_range(a, r);
  const int kbeg = split * a.split_keys;
  const int kend = min(kbeg + a.split_keys, rr.end);
  if (a.nsplit > 1 && kbeg >= rr.end) return;  // empty split: the merge skips it

  // this lane's query row (MFMA column)
  const int rows_kv = a.N * a.g;
  const int rho = qb * kRowsPerBlock + wave * kRowsPerWave + col;
  const bool row_in = rho < rows_kv;
  const int node = row_in ? rho / a.g : 0;
  const int hq = kvh * a.g + (row_in ? rho % a.g : 0);
  const bool row_live = row_in && node < rr.cnt;

  // Q^T fragments: 8 consecutive d of the lane's row per contraction step
  u32x4 bq[KS];
  {
    const uint16_t* qrow = a.q + (((size_t)r * a.N + node) * a.Hq + hq) * D + grp * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_live) v = *(const u32x4*)(qrow + s * 32);
      bq[s] = v;
    }
  }
  const uint32_t* mrow = a.mask + ((size_t)r * a.N + node) * a.NW;

  f32x4 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = kNegInf, l = 0.0f;

  // cooperative staging: thread -> (key, 8 d) for K, (key pair, 8 d) for V
  const int st_key = tid >> 4;          // 0..15
  const int st_d = (tid & 15) * 8;      // first d of the thread's group
  constexpr int DG = D / 8;             // 16-byte groups per row
  const size_t kvbase = ((size_t)r * a.Hkv + kvh) * a.C;
  const uint16_t* kbase_p = a.k + kvbase * D;
  const uint16_t* vbase_p = a.v + kvbase * D;

  // registers of the next chunk: K rows st_key and st_key + 16, V rows of the
  // pair (2 st_key, 2 st_key + 1), 8 d each; for D = 64 only the threads with
  // a d group below 8 stage.
  u32x4 nk0, nk1, nv0, nv1;
  const bool st_on = (tid & 15) < DG;
  auto fetch = [&](int c0) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    nk0 = z;
    nk1 = z;
    nv0 = z;
    nv1 = z;
    if (!st_on) return;
    const int s0 = c0 + st_key, s1 = c0 + st_key + 16;
    if (s0 < kend) nk0 = *(const u32x4*)(kbase_p + (size_t)s0 * D + st_d);
    if (s1 < kend) nk1 = *(const u32x4*)(kbase_p + (size_t)s1 * D + st_d);
    const int v0 = c0 + 2 * st_key, v1 = v0 + 1;
    if (v0 < kend) nv0 = *(const u32x4*)(vbase_p + (size_t)v0 * D + st_d);
    if (v1 < kend) nv1 = *(const u32x4*)(vbase_p + (size_t)v1 * D + st_d);
  };
  auto stage = [&]() {
    if (!st_on) return;
    *(u32x4*)(sK + st_key * KROW + st_d) = nk0;
    *(u32x4*)(sK + (st_key + 16) * KROW + st_d) = nk1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t lo = nv0[i], hi = nv1[i];
      // d = st_d + 2i and st_d + 2i + 1; keys 2 st_key (low half), 2 st_key + 1
      *(uint32_t*)(sV + (st_d + 2 * i) * VROW + 2 * st_key) = (lo & 0xffffu) | (hi << 16);
      *(uint32_t*)(sV + (st_d + 2 * i + 1) * VROW + 2 * st_key) = (lo >> 16) | (hi & 0xffff0000u);
    }
  };

  // A-operand rows of the S^T tile pair: tile 0 holds keys 8c + e, tile 1 keys
  // 8c + 4 + e, for MFMA row 4c + e (c = col / 4, e = col % 4)
  const int krow0 = 8 * (col >> 2) + (col & 3);
  const int krow1 = krow0 + 4;

  if (kbeg < kend) fetch(kbeg);
  for (int c0 = kbeg; c0 < kend; c0 += kChunk) {
    __syncthreads();  // the previous chunk is no longer read
    stage();
    __syncthreads();
    if (c0 + kChunk < kend) fetch(c0 + kChunk);

    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 a0 = *(const u32x4*)(sK + krow0 * KROW + s * 32 + grp * 8);
      const u32x4 a1 = *(const u32x4*)(sK + krow1 * KROW + s * 32 + grp * 8);
      s0 = mfma_bf16(a0, bq[s], s0);
      s1 = mfma_bf16(a1, bq[s], s1);
    }
    // the lane's 8 keys: slot c0 + 8 grp + i, i = 0..7
    float sc[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sc[e] = s0[e] * a.scale_log2;
      sc[4 + e] = s1[e] * a.scale_log2;
    }
    const int kfirst = c0 + 8 * grp;
    bool ok[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int slot = kfirst + i;
      bool adm = row_live && slot < kend;
      if (adm && slot >= rr.prefix) {
        const int j = slot - rr.prefix;  // tree node j < count
        adm = (mrow[j >> 5] >> (j & 31)) & 1u;
      }
      ok[i] = adm;
    }
    float cmax = kNegInf;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (ok[i]) cmax = fmaxf(cmax, sc[i]);
    cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
    cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
    const float mn = fmaxf(m, cmax);
    float p[8];
    float alpha = 1.0f;
    if (mn == kNegInf) {
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = 0.0f;
    } else {
      alpha = exp2_hw(m - mn);  // m = -inf gives 0 (nothing accumulated yet)
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = ok[i] ? exp2_hw(sc[i] - mn) : 0.0f;
    }
    m = mn;
    float ps = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ps += p[i];
    l = l * alpha + ps;
    u32x4 bp;
#pragma unroll
    for (int i = 0; i < 4; ++i) bp[i] = bf16_rne_bits(p[2 * i]) | (bf16_rne_bits(p[2 * i + 1]) << 16);
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const u32x4 av = *(const u32x4*)(sV + (t * 16 + col) * VROW + 8 * grp);
      o[t] = mfma_bf16(av, bp, o[t] * alpha);
    }
  }

  // the row's sum over its four lane groups
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (!row_in) return;
  const size_t qidx = ((size_t)r * a.N + node) * a.Hq + hq;  // (request, node, head)
  if (a.nsplit == 1) {
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
    uint16_t* orow = a.out + qidx * D;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const f32x4 v = o[t] * inv;
      u32x2 w;
      w[0] = bf16_rne_bits(v[0]) | (bf16_rne_bits(v[1]) << 16);
      w[1] = bf16_rne_bits(v[2]) | (bf16_rne_bits(v[3]) << 16);
      *(u32x2*)(orow + t * 16 + 4 * grp) = w;
    }
  } else {
    const size_t prow = (size_t)split * a.R * a.N * a.Hq + qidx;
    float* po = a.part_o + prow * D;
#pragma unroll
    for (int t = 0; t < DT; ++t) *(f32x4*)(po + t * 16 + 4 * grp) = o[t];
    if (grp == 0) {
      a.part_ml[2 * prow] = m;
      a.part_ml[2 * prow + 1] = l;
    }
  }
}

// Merge of the split runs: one thread per (row, d), rows of (request, node,
// head).  Only the splits that hold admitted slots were written.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_merge_kernel(AttnArgs a) {
  constexpr int RPB = kThreads / D;  // rows per workgroup
  const size_t rows = (size_t)a.R * a.N * a.Hq;
  const size_t qidx = (size_t)blockIdx.x * RPB + threadIdx.x / D;
  const int d = threadIdx.x % D;
  if (qidx >= rows) return;
  const int r = (int)(qidx / ((size_t)a.N * a.Hq));
  const int node = (int)(qidx / a.Hq % a.N);
  const ReqRange rr = req_range(a, r);
  float val = 0.0f;
  if (node < rr.cnt && rr.end > 0) {
    const int ns = min(a.nsplit, (rr.end + a.split_keys - 1) / a.split_keys);
    float M = kNegInf;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, a.part_ml[2 * ((size_t)s * rows + qidx)]);
    if (M != kNegInf) {
      float L = 0.0f, O = 0.0f;
      for (int s = 0; s < ns; ++s) {
        const size_t prow = (size_t)s * rows + qidx;
        const float ms = a.part_ml[2 * prow];
        if (ms == kNegInf) continue;  // no admitted slot of this row in split s
        const float w = exp2_hw(ms - M);
        L += w * a.part_ml[2 * prow + 1];
        O += w * a.part_o[prow * D + d];
      }
      val = L > 0.0f ? O / L : 0.0f;
    }
  }
  a.out[qidx * D + d] = (uint16_t)bf16_rne_bits(val);
}

}  // namespace

AttnPlan plan_attention(int R, int N, int Hq, int Hkv, int D, int C, int cus) {
  AttnPlan p;
  const int g = Hq / Hkv;
  p.qblocks = (N * g + kRowsPerBlock - 1) / kRowsPerBlock;
  const long long base = (long long)R * Hkv * p.qblocks;
  const int chunks = (C + kChunk - 1) / kChunk;
  int ns = 1;
  if (base < 2LL * cus) ns = (int)((2LL * cus + base - 1) / base);
  ns = ns < chunks ? ns : chunks;
  ns = ns < 1 ? 1 : ns;
  const int per = (chunks + ns - 1) / ns;  // chunks per split
  p.split_keys = per * kChunk;
  p.nsplit = (chunks + per - 1) / per;
  const size_t rows = (size_t)R * N * Hq;
  p.ws_bytes = p.nsplit > 1 ? (size_t)p.nsplit * rows * (D + 2) * sizeof(float) + 256 : 0;
  return p;
}

hipError_t launch_attention(AttnArgs a, int D, hipStream_t stream) {
  const dim3 grid(a.qblocks * a.nsplit, a.Hkv, a.R);
  if (D == 128)
    attn_kernel<128><<<grid, kThreads, 0, stream>>>(a);
  else
    attn_kernel<64><<<grid, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  const size_t rows = (size_t)a.R * a.N * a.Hq;
  const int rpb = kThreads / D;
  const unsigned blocks = (unsigned)((rows + rpb - 1) / rpb);
  if (D == 128)
    attn_merge_kernel<128><<<blocks, kThreads, 0, stream>>>(a);
  else
    attn_merge_kernel<64><<<blocks, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace pctree

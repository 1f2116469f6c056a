// C ABI of the PCTree tree builder: argument checking, workspace layout and
// the launch sequence.  Every check runs on the host before anything is
// enqueued, so an error status means no device work was issued.
#include "pctree.h"

#include <algorithm>
#include <mutex>

#include "pctree_attention.h"
#include "pctree_plan.h"
#include "pctree_verify.h"

namespace pctree {

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int pow2ceil(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr & (a - 1)) == 0; }

pctree_status check_shape(const pctree_shape* s) {
  if (!s) return PCTREE_ERR_INVALID_ARGUMENT;
  if (s->vocab < 1 || s->block < 1 || s->budget < 1 || s->topk < 1 || s->rank < 1 ||
      s->requests < 1)
    return PCTREE_ERR_INVALID_ARGUMENT;
  if (s->dtype != PCTREE_F32 && s->dtype != PCTREE_BF16) return PCTREE_ERR_INVALID_ARGUMENT;
  if (s->mode < 0 || s->mode > 2) return PCTREE_ERR_UNSUPPORTED;
  if (s->vocab > PCTREE_MAX_VOCAB || s->block > PCTREE_MAX_BLOCK || s->topk > PCTREE_MAX_TOPK ||
      s->budget > PCTREE_MAX_BUDGET || s->requests > PCTREE_MAX_REQUESTS)
    return PCTREE_ERR_UNSUPPORTED;
  if (s->dtype == PCTREE_BF16 && (s->rank % 32 != 0 || s->rank > PCTREE_MAX_RANK_BF16))
    return PCTREE_ERR_UNSUPPORTED;
  if (s->dtype == PCTREE_F32 && (s->rank % 16 != 0 || s->rank > PCTREE_MAX_RANK_F32))
    return PCTREE_ERR_UNSUPPORTED;
  return PCTREE_OK;
}

pctree_status check_inputs(const pctree_inputs* in) {
  if (!in || !in->base_logits || !in->emb || !in->proj_t || !in->depth_feat || !in->root_token ||
      !in->prefix_len)
    return PCTREE_ERR_INVALID_ARGUMENT;
  if (!aligned(in->base_logits, 16) || !aligned(in->emb, 16) || !aligned(in->proj_t, 16) ||
      !aligned(in->depth_feat, 16) || !aligned(in->root_token, 4) || !aligned(in->prefix_len, 4))
    return PCTREE_ERR_INVALID_ARGUMENT;
  return PCTREE_OK;
}

// Tree attention: shape checks and the work split.  The split is planned for
// the 256 compute units of the gfx950 part, so that the workspace size is a
// function of the shape alone.
constexpr int kAttnPlanCUs = 256;

pctree_status check_attn_shape(const pctree_attn_shape* s) {
  if (!s) return PCTREE_ERR_INVALID_ARGUMENT;
  if (s->requests < 1 || s->budget < 1 || s->q_heads < 1 || s->kv_heads < 1 ||
      s->head_dim < 1 || s->capacity < 1)
    return PCTREE_ERR_INVALID_ARGUMENT;
  if (s->q_heads % s->kv_heads != 0) return PCTREE_ERR_INVALID_ARGUMENT;
  if (!(s->scale > 0.0f) || s->scale > 3.4e38f)
    return PCTREE_ERR_INVALID_ARGUMENT;  // scale not positive and finite
  if (s->head_dim != 64 && s->head_dim != 128) return PCTREE_ERR_UNSUPPORTED;
  if (s->budget > PCTREE_MAX_MASK_BUDGET || s->requests > 65535 || s->kv_heads > 65535)
    return PCTREE_ERR_UNSUPPORTED;
  // element counts of q / out and of one cache tensor stay far inside size_t,
  // and the grid (groups x query blocks, padded to whole XCD rounds) inside int
  const long long rows = (long long)s->requests * s->budget * s->q_heads;
  const long long slots = (long long)s->requests * s->kv_heads * s->capacity;
  if (rows > (1LL << 31) / s->head_dim || slots > (1LL << 40) / s->head_dim)
    return PCTREE_ERR_UNSUPPORTED;
  return PCTREE_OK;
}

AttnPlan attn_plan(const pctree_attn_shape* s) {
  return plan_attention(s->requests, s->budget, s->q_heads, s->kv_heads, s->head_dim,
                        s->capacity, kAttnPlanCUs);
}

// Chain decode runs the tree builder with k = 1 and N = B + 1; its tree
// outputs other than tokens and log-probabilities live in the workspace.
struct ChainScratch {
  size_t parent, depth, position, count, total;
};

ChainScratch chain_scratch(int R, int B) {
  ChainScratch c;
  const size_t row = align256((size_t)R * (B + 1) * sizeof(int32_t));
  c.parent = 0;
  c.depth = row;
  c.position = 2 * row;
  c.count = 3 * row;
  c.total = 3 * row + align256((size_t)R * sizeof(int32_t));
  return c;
}

size_t tree_bytes(const pctree_shape* s) {
  Plan p{};
  plan_shape(p, s->vocab, s->block, s->budget, s->topk, s->rank, s->requests, s->dtype);
  return carve_workspace(p, nullptr);
}

size_t chain_bytes(const pctree_shape* s) {
  Plan p{};
  plan_shape(p, s->vocab, s->block, s->block + 1, 1, s->rank, s->requests, s->dtype);
  return carve_workspace(p, nullptr) + chain_scratch(s->requests, s->block).total;
}

void bind_inputs(Plan& p, const pctree_inputs* in) {
  p.L = in->base_logits;
  p.E = in->emb;
  p.Wt = in->proj_t;
  p.h = in->depth_feat;
  p.root = in->root_token;
  p.prefix = in->prefix_len;
}

pctree_status enqueue(const Plan& p, void* stream) {
  (void)hipGetLastError();  // start from a clean error state
  const hipError_t e = launch_round(p, (hipStream_t)stream);
  return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
}

// The checks of pctree_build_tree that do not concern the workspace.
pctree_status check_tree_args(const pctree_shape* shape, const pctree_inputs* in,
                              const pctree_tree* out, const pctree_trace* trace) {
  pctree_status st = check_shape(shape);
  if (st != PCTREE_OK) return st;
  if ((st = check_inputs(in)) != PCTREE_OK) return st;
  if (!out || !out->token || !out->parent || !out->depth || !out->position || !out->logprob ||
      !out->count)
    return PCTREE_ERR_INVALID_ARGUMENT;
  if (!aligned(out->token, 4) || !aligned(out->parent, 4) || !aligned(out->depth, 4) ||
      !aligned(out->position, 4) || !aligned(out->logprob, 4) || !aligned(out->count, 4) ||
      !aligned(out->mask, 4))
    return PCTREE_ERR_INVALID_ARGUMENT;
  if (trace && (!trace->token || !trace->parent_slot || !trace->score ||
                !aligned(trace->token, 4) || !aligned(trace->parent_slot, 4) ||
                !aligned(trace->score, 4)))
    return PCTREE_ERR_INVALID_ARGUMENT;
  return PCTREE_OK;
}

// Enqueue one round of a checked call on a workspace of at least
// tree_bytes(shape) bytes at `ws` (256-byte aligned).
pctree_status enqueue_tree(const pctree_shape* shape, const pctree_inputs* in,
                           const pctree_tree* out, const pctree_trace* trace, char* ws,
                           void* stream) {
  Plan p{};
  plan_shape(p, shape->vocab, shape->block, shape->budget, shape->topk, shape->rank,
             shape->requests, shape->dtype);
  carve_workspace(p, ws);
  bind_inputs(p, in);
  p.mode = shape->mode;
  p.o_token = out->token;
  p.o_parent = out->parent;
  p.o_depth = out->depth;
  p.o_position = out->position;
  p.o_logprob = out->logprob;
  p.o_count = out->count;
  p.o_mask = out->mask;
  p.t_token = trace ? trace->token : nullptr;
  p.t_pslot = trace ? trace->parent_slot : nullptr;
  p.t_score = trace ? trace->score : nullptr;
  return enqueue(p, stream);
}

// ---------------------------------------------------------------------------
// Workspace of pctree_build_tree_noalloc: a fixed array in device memory, one
// copy per device, held until the process ends.  In host code `scratch`
// names a host-side stand-in, not device memory: its device address is
// looked up once per device (with that device current) and only that
// address is ever passed to a kernel.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = PCTREE_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipErrorUnknown;
};

ScratchSlot g_scratch[kMaxDevices];

// Device address of the current device's scratch array (nullptr on failure).
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  ScratchSlot& s = g_scratch[dev];
  std::call_once(s.once, [&s] {
    void* ptr = nullptr;
    s.err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    s.ptr = s.err == hipSuccess ? ptr : nullptr;
  });
  return s.ptr;
}

}  // namespace

void plan_shape(Plan& p, int V, int B, int N, int k, int r, int R, int dtype) {
  p.V = V;
  p.B = B;
  p.N = N;
  p.k = k;
  p.kk = std::min(k, V);
  p.r = r;
  p.R = R;
  p.dtype = dtype;
  p.kmax = pow2ceil(p.kk);
  p.nchunk = dtype ? r / 32 : r / 16;
  p.ntiles = (V + kTile - 1) / kTile;
  // multi-launch form: about one slice per CU of a 256-CU device (the
  // persistent form sizes its slices from the device at launch)
  p.tiles_per_slice = std::max(4, (p.ntiles + 255) / 256);
  p.G = (p.ntiles + p.tiles_per_slice - 1) / p.tiles_per_slice;
  p.maxpool = 1 + p.kk + (B - 1) * p.kk * p.kk;
  p.rows_max = R * p.kk;
  // the persistent form keeps every stage's partials (blocks read them while
  // others already publish the next stage); the multi-launch form reuses one
  p.stages = p.rows_max <= kNarrowRows ? B : 1;
}

size_t carve_workspace(Plan& p, char* base) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* ptr = base ? base + off : nullptr;
    off += align256(bytes);
    return ptr;
  };
  const size_t R = p.R, kk = p.kk, es = p.dtype ? 2 : 4;
  p.U = take(R * kk * p.r * es);
  p.front_node = (int*)take(R * kk * sizeof(int));
  p.front_tok = (int*)take(R * kk * sizeof(int));
  p.front_score = (float*)take(R * kk * sizeof(float));
  p.node_tok = (int*)take(R * p.maxpool * sizeof(int));
  p.node_par = (int*)take(R * p.maxpool * sizeof(int));
  p.node_depth = (int*)take(R * p.maxpool * sizeof(int));
  p.node_score = (float*)take(R * p.maxpool * sizeof(float));
  p.top_key = (uint64_t*)take(R * p.N * sizeof(uint64_t));
  p.top_node = (int*)take(R * p.N * sizeof(int));
  const size_t parts = (size_t)p.stages * p.rows_max * kSlicesMax;
  p.part_key = (uint64_t*)take(parts * p.kmax * sizeof(uint64_t));
  p.part_hd = (uint64_t*)take(parts * kRecWords * sizeof(uint64_t));
  p.req_bad = (int*)take(R * sizeof(int));
  p.front_w = (uint64_t*)take((size_t)p.stages * p.rows_max * sizeof(uint64_t));
  p.tau = (float*)take((size_t)p.rows_max * sizeof(float));
  p.probe_tok = (int*)take(R * (size_t)p.B * kProbe * sizeof(int));
  p.probe_w = take(R * (size_t)p.B * kProbe * p.r * es);
  p.probe_l = (float*)take(R * (size_t)p.B * kProbe * sizeof(float));
  p.thr_ms = (float*)take((size_t)p.rows_max * kSlicesMax * 2 * sizeof(float));
  p.thr_cnt = (int*)take((size_t)p.rows_max * kSlicesMax * sizeof(int));
  return off;
}

}  // namespace pctree

using namespace pctree;

extern "C" {

size_t pctree_workspace_bytes(const pctree_shape* shape) {
  if (check_shape(shape) != PCTREE_OK) return 0;
  return std::max(tree_bytes(shape), chain_bytes(shape));
}

pctree_status pctree_build_tree(const pctree_shape* shape, const pctree_inputs* in,
                                const pctree_tree* out, const pctree_trace* trace,
                                void* workspace, size_t workspace_bytes, void* stream) {
  try {
    const pctree_status st = check_tree_args(shape, in, out, trace);
    if (st != PCTREE_OK) return st;
    if (!workspace || !aligned(workspace, 256)) return PCTREE_ERR_WORKSPACE;
    if (workspace_bytes < tree_bytes(shape)) return PCTREE_ERR_WORKSPACE;
    return enqueue_tree(shape, in, out, trace, (char*)workspace, stream);
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_build_tree_noalloc(const pctree_shape* shape, const pctree_inputs* in,
                                        const pctree_tree* out, const pctree_trace* trace,
                                        void* stream) {
  try {
    const pctree_status st = check_tree_args(shape, in, out, trace);
    if (st != PCTREE_OK) return st;
    // checked before any HIP call: a shape past the array's size is an error
    if (tree_bytes(shape) > kScratchBytes) return PCTREE_ERR_WORKSPACE;
    char* ws = (char*)scratch_address();
    if (!ws) return PCTREE_ERR_HIP;
    // the round clears every word it polls before use, so what an earlier
    // call left in the array does not matter
    return enqueue_tree(shape, in, out, trace, ws, stream);
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_build_mask(const int32_t* parent, const int32_t* count, int32_t requests,
                                int32_t budget, uint32_t* mask, void* stream) {
  try {
    if (!parent || !count || !mask || requests < 1 || budget < 1)
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (!aligned(parent, 4) || !aligned(count, 4) || !aligned(mask, 4))
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (budget > PCTREE_MAX_MASK_BUDGET || requests > 65535) return PCTREE_ERR_UNSUPPORTED;
    (void)hipGetLastError();
    const hipError_t e = launch_mask(parent, count, requests, budget, mask, (hipStream_t)stream);
    return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_chain_decode(const pctree_shape* shape, const pctree_inputs* in,
                                  int32_t* chain_token, float* chain_logprob, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  try {
    if (!shape) return PCTREE_ERR_INVALID_ARGUMENT;
    pctree_shape cs = *shape;
    cs.topk = 1;
    cs.budget = std::max(1, std::min(shape->block, PCTREE_MAX_BLOCK) + 1);
    pctree_status st = check_shape(&cs);
    if (st != PCTREE_OK) return st;
    if ((st = check_inputs(in)) != PCTREE_OK) return st;
    if (!chain_token || !chain_logprob || !aligned(chain_token, 4) || !aligned(chain_logprob, 4))
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (!workspace || !aligned(workspace, 256)) return PCTREE_ERR_WORKSPACE;
    if (workspace_bytes < chain_bytes(&cs)) return PCTREE_ERR_WORKSPACE;

    Plan p{};
    plan_shape(p, cs.vocab, cs.block, cs.budget, 1, cs.rank, cs.requests, cs.dtype);
    const size_t tb = carve_workspace(p, (char*)workspace);
    const ChainScratch c = chain_scratch(cs.requests, cs.block);
    char* sb = (char*)workspace + tb;
    bind_inputs(p, in);
    p.mode = shape->mode;
    p.o_token = chain_token;
    p.o_logprob = chain_logprob;
    p.o_parent = (int*)(sb + c.parent);
    p.o_depth = (int*)(sb + c.depth);
    p.o_position = (int*)(sb + c.position);
    p.o_count = (int*)(sb + c.count);
    p.o_mask = nullptr;
    p.t_token = nullptr;
    p.t_pslot = nullptr;
    p.t_score = nullptr;
    return enqueue(p, stream);
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_build_retrieve(const int32_t* parent, const int32_t* count, int32_t requests,
                                    int32_t budget, int32_t max_depth, int32_t* rows,
                                    int32_t* nrows, void* stream) {
  try {
    if (!parent || !count || !rows || !nrows || requests < 1 || budget < 1 || max_depth < 0)
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (!aligned(parent, 4) || !aligned(count, 4) || !aligned(rows, 4) || !aligned(nrows, 4))
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (budget > PCTREE_MAX_MASK_BUDGET || max_depth > PCTREE_MAX_BLOCK || requests > 65535)
      return PCTREE_ERR_UNSUPPORTED;
    (void)hipGetLastError();
    const hipError_t e = launch_retrieve(parent, count, requests, budget, max_depth + 1, rows,
                                         nrows, (hipStream_t)stream);
    return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_accept_greedy(const int32_t* token, const int32_t* rows,
                                   const int32_t* nrows, const int32_t* target_next,
                                   int32_t requests, int32_t budget, int32_t max_depth,
                                   int32_t* accept_len, int32_t* accept_row,
                                   int32_t* accept_node, int32_t* bonus, void* stream) {
  try {
    if (!token || !rows || !nrows || !target_next || !accept_len || !accept_row ||
        !accept_node || !bonus || requests < 1 || budget < 1 || max_depth < 0)
      return PCTREE_ERR_INVALID_ARGUMENT;
    for (const void* q : {(const void*)token, (const void*)rows, (const void*)nrows,
                          (const void*)target_next, (const void*)accept_len,
                          (const void*)accept_row, (const void*)accept_node, (const void*)bonus})
      if (!aligned(q, 4)) return PCTREE_ERR_INVALID_ARGUMENT;
    if (budget > PCTREE_MAX_MASK_BUDGET || max_depth > PCTREE_MAX_BLOCK || requests > 65535)
      return PCTREE_ERR_UNSUPPORTED;
    (void)hipGetLastError();
    const hipError_t e = launch_accept(token, rows, nrows, target_next, requests, budget,
                                       max_depth + 1, accept_len, accept_row, accept_node, bonus,
                                       (hipStream_t)stream);
    return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

pctree_status pctree_compact_kv(void* cache, int64_t request_stride, int64_t group_stride,
                                int32_t groups, int32_t capacity, int32_t slot_bytes,
                                const int32_t* prefix_len, const int32_t* accept_node,
                                const int32_t* accept_len, int32_t requests, int32_t budget,
                                int32_t max_depth, void* stream) {
  try {
    if (!cache || !prefix_len || !accept_node || !accept_len || requests < 1 || budget < 1 ||
        max_depth < 0 || groups < 1 || capacity < 1 || slot_bytes < 16)
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (!aligned(cache, 16) || slot_bytes % 16 != 0 || request_stride % 16 != 0 ||
        group_stride % 16 != 0 || request_stride < 0 || group_stride < 0 ||
        !aligned(prefix_len, 4) || !aligned(accept_node, 4) || !aligned(accept_len, 4))
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (max_depth > PCTREE_MAX_BLOCK || requests > 65535 || budget > PCTREE_MAX_MASK_BUDGET)
      return PCTREE_ERR_UNSUPPORTED;
    // the grid covers groups x (slot_bytes / 16) columns per request
    if ((long long)groups * (slot_bytes / 16) > (long long)INT32_MAX)
      return PCTREE_ERR_UNSUPPORTED;
    (void)hipGetLastError();
    const hipError_t e = launch_compact(cache, request_stride, group_stride, groups, capacity,
                                        slot_bytes, prefix_len, accept_node, accept_len, requests,
                                        budget, max_depth + 1, (hipStream_t)stream);
    return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

size_t pctree_attention_workspace_bytes(const pctree_attn_shape* shape) {
  if (check_attn_shape(shape) != PCTREE_OK) return 0;
  return attn_plan(shape).ws_bytes;
}

pctree_status pctree_tree_attention(const pctree_attn_shape* shape, const void* q,
                                    const void* k_cache, const void* v_cache,
                                    const uint32_t* mask, const int32_t* count,
                                    const int32_t* prefix_len, void* out, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  try {
    const pctree_status st = check_attn_shape(shape);
    if (st != PCTREE_OK) return st;
    if (!q || !k_cache || !v_cache || !mask || !count || !prefix_len || !out)
      return PCTREE_ERR_INVALID_ARGUMENT;
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
        !aligned(mask, 4) || !aligned(count, 4) || !aligned(prefix_len, 4))
      return PCTREE_ERR_INVALID_ARGUMENT;
    const AttnPlan plan = attn_plan(shape);
    if (plan.ws_bytes > 0 &&
        (!workspace || !aligned(workspace, 256) || workspace_bytes < plan.ws_bytes))
      return PCTREE_ERR_WORKSPACE;
    AttnArgs a;
    a.q = (const uint16_t*)q;
    a.k = (const uint16_t*)k_cache;
    a.v = (const uint16_t*)v_cache;
    a.mask = mask;
    a.count = count;
    a.prefix_len = prefix_len;
    a.out = (uint16_t*)out;
    a.R = shape->requests;
    a.N = shape->budget;
    a.Hq = shape->q_heads;
    a.Hkv = shape->kv_heads;
    a.C = shape->capacity;
    a.NW = (shape->budget + 31) / 32;
    a.g = shape->q_heads / shape->kv_heads;
    a.qblocks = plan.qblocks;
    a.nsplit = plan.nsplit;
    a.split_keys = plan.split_keys;
    a.scale_log2 = shape->scale * 1.4426950408889634f;
    const size_t rows = (size_t)a.R * a.N * a.Hq;
    a.part_o = plan.nsplit > 1 ? (float*)workspace : nullptr;
    a.part_ml = plan.nsplit > 1 ? (float*)workspace + (size_t)plan.nsplit * rows * shape->head_dim
                                : nullptr;
    (void)hipGetLastError();
    const hipError_t e = launch_attention(a, plan.blocks, shape->head_dim, (hipStream_t)stream);
    return e == hipSuccess ? PCTREE_OK : PCTREE_ERR_HIP;
  } catch (...) {
    return PCTREE_ERR_HIP;
  }
}

const char* pctree_status_string(pctree_status status) {
  switch (status) {
    case PCTREE_OK: return "PCTREE_OK";
    case PCTREE_ERR_INVALID_ARGUMENT: return "PCTREE_ERR_INVALID_ARGUMENT";
    case PCTREE_ERR_UNSUPPORTED: return "PCTREE_ERR_UNSUPPORTED";
    case PCTREE_ERR_WORKSPACE: return "PCTREE_ERR_WORKSPACE";
    case PCTREE_ERR_HIP: return "PCTREE_ERR_HIP";
  }
  return "PCTREE_ERR_UNKNOWN";
}

int32_t pctree_abi_version(void) { return PCTREE_ABI_VERSION; }

}  // extern "C"

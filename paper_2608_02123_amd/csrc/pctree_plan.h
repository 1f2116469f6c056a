// Internal launch plan shared by the C ABI (pctree_api.hip) and the kernels
// (pctree_kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pctree {

constexpr int kTile = 16;           // tokens per MFMA output tile (M of 16x16xK)
constexpr int kSlicesMax = 512;     // V-slices of one head launch
constexpr int kRoundSlicesMax = 256;  // V-slices of the persistent round kernel
constexpr int kHeadThreads = 256;   // 4 waves
constexpr int kSelectThreads = 1024;
constexpr int kEmitThreads = 256;
constexpr int kMaskThreads = 256;
constexpr int kRoundWaves = 8;       // waves per WG of the persistent round kernel
constexpr int kNarrowRows = 16;      // frontier rows (R * k') one column block holds
constexpr int kFlagStride = 64;      // ints between two workgroups' flag words (256 B)
constexpr int kProbe = 32;           // probe tokens per (request, depth) of the wide stages

// What a streaming workgroup publishes per (stage, row, slice) besides its
// candidate list, the slice record: kRecWords 64-bit words, the list's
// kHeadKeys best keys (0 past the list) and the slice's sum of exp relative to
// its best logit (the logit of the first key) in the low half of the last
// word.  Records are stored word-major, [stage][row][word][slice], so that a
// wave reads one word of 64 slices as 512 contiguous bytes.  Every published
// word carries the call's tag (the low kTagBits of a key, the high half of the
// sum word), so that a reader can tell a word of this call from a stale one
// without any ordering between words.
constexpr int kHeadKeys = 3;
constexpr int kRecWords = kHeadKeys + 1;
constexpr int kTagBits = 10;
constexpr uint32_t kTagMask = (1u << kTagBits) - 1;

// Everything one round needs, passed by value to every kernel.
struct Plan {
  // problem size
  int V, B, N, k, kk, r, R, dtype;  // kk = min(k, V); dtype 0 = f32, 1 = bf16
  int kmax;                         // per-row candidate list length: pow2 >= kk
  int nchunk;                       // 16-byte rank chunks per row: r/32 (bf16), r/16 (f32)
  int G, tiles_per_slice, ntiles;   // head-stream V-slicing
  int maxpool;                      // 1 + kk + (B-1) kk^2
  int rows_max;                     // R * kk
  int stages;                       // stages with their own partial buffers (B, or 1)

  // inputs
  const void* L;
  const void* E;
  const void* Wt;
  const float* h;
  const int* root;
  const int* prefix;

  // outputs
  int* o_token;
  int* o_parent;
  int* o_depth;
  int* o_position;
  int* o_count;
  float* o_logprob;
  uint32_t* o_mask;  // may be null
  int* t_token;      // trace, may be null
  int* t_pslot;
  float* t_score;

  // workspace
  void* U;           // [R][kk][r] head activations of the current frontier (dtype)
  int* front_node;   // [R][kk] pool id of each frontier slot
  int* front_tok;    // [R][kk]
  float* front_score;// [R][kk]
  int* node_tok;     // [R][maxpool] candidate pool
  int* node_par;     // [R][maxpool] pool id of the parent
  int* node_depth;   // [R][maxpool]
  float* node_score; // [R][maxpool]
  uint64_t* top_key; // [R][N] running global top-N (sorted, descending)
  int* top_node;     // [R][N]
  uint64_t* part_key;// [stages][rows_max][kSlicesMax][kmax] per-slice candidate lists
  uint64_t* part_hd; // [stages][rows_max][kRecWords][kSlicesMax] slice records
  int* req_bad;      // [R] root token outside [0, V)
  uint64_t* front_w; // [stages][rows_max] frontier of each stage (persistent form)
  float* tau;        // [rows_max] wide stages: lower bound of each row's k'-th best logit
  int* probe_tok;    // [R][B][kProbe] wide stages: probe tokens of each request and depth
  void* probe_w;     // [R][B][kProbe][r] (dtype) their W rows (zero for a missing probe)
  float* probe_l;    // [R][B][kProbe] their base logits L_d
  float* thr_ms;     // [rows_max][kSlicesMax][2] wide stages: each slice's (max, sum of exp)
  int* thr_cnt;      // [rows_max][kSlicesMax] wide stages: candidates each slice kept
  uint32_t tag;      // this call's tag, 1 .. kTagMask (published words carry it)
  int mode;          // 0 parent-conditioned, 1 Shared-Markov, 2 parent-independent
  int unbounded;     // wide stages ignore tau (every logit is a candidate)
  long long spin_ticks;  // device wall-clock ticks a wait may last before aborting
  int lds_tiles;         // W tiles a streaming block keeps in LDS for the whole round
  int lds_top_offset;    // byte offset of the keeper's running top-N in the dynamic LDS
  int lds_tile_offset;   // byte offset of the resident W tiles in the dynamic LDS
};

// Workspace layout for a plan; offsets are 256-byte aligned.  With base ==
// nullptr only the total is computed.
size_t carve_workspace(Plan& p, char* base);

// Fill the shape-derived fields of a plan (no pointers).
void plan_shape(Plan& p, int V, int B, int N, int k, int r, int R, int dtype);

// Enqueue one full round on `stream`.
hipError_t launch_round(const Plan& p, hipStream_t stream);

// Process-wide diagnostic overrides of the launch (pctree_debug_set in
// include/pctree_profile.h); the defaults leave every launch as planned.
struct DebugConfig {
  long long wait_ticks = -1;  // < 0: 2 s of device wall clock per bounded wait
  int force_multilaunch = 0;  // nonzero: per-stage launches even for narrow rounds
  int round_slices = 0;       // > 0: V-slices of the persistent round (else one per CU but one)
  int wide_unbounded = 0;     // nonzero: wide stages without their per-row bound
};
DebugConfig& debug_config();

// Event bracketing of the dominant kernel (pctree_profile.hip): call
// profile_mark() right before and right after each of its launches.
bool profile_on();
void profile_mark(hipStream_t stream, const char* kernel);

// Stage timeline of the diagnostic build (compiled with PCTREE_TIMELINE):
// [who][stage][event] device wall-clock stamps (include/pctree_profile.h
// lists the workgroups and events).  timeline_copy copies them to `host`
// (when not null) and then zeroes them if `clear`; hipErrorNotSupported in
// the default build, which has no stamps.
constexpr int kTimelineWho = 5, kTimelineStages = 65, kTimelineEvents = 8;
bool timeline_built();
hipError_t timeline_copy(long long* host, bool clear);

// Enqueue the standalone ancestor-mask kernel.
hipError_t launch_mask(const int* parent, const int* count, int R, int N, uint32_t* mask,
                       hipStream_t stream);

}  // namespace pctree

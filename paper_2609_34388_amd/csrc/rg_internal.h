// Internal launch-side structures shared by the host API and the kernels.
// Not part of the public ABI (include/recguide.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace rg {

constexpr int kPageSize = 16;
constexpr int kMaxReqPerLaunch = 128;  // equals RG_ATTN_MAX_REQS_PER_LAUNCH
constexpr int kKeyTile = 128;          // keys per LDS buffer; chunks are multiples of it
constexpr int kMaxChunkKeys = 1 << 16;  // keys per work item at most
constexpr int kSyncHeader = 4;          // queue head, exit count, give-up flag, report word
// Combine items of one launch the one-launch kernel can count (two counters
// each); launches with more use the main kernel plus the combine kernel.
constexpr int kMaxSyncComb = 16384;
// The synchronisation words open every attention workspace at a fixed place
// and size, so calls with different layouts can share a workspace: the words
// one call leaves at zero are never another call's partials.
constexpr int kSyncWords = kSyncHeader + 2 * kMaxSyncComb;

// Per-request data of one attention launch.  Everything a work group needs
// about its request travels in the kernel arguments, so no table has to be
// copied to the device before the kernels run.
struct AttnReq {
  int32_t q_start;     // first query row (token) of the request
  int32_t ctx;         // cached context tokens L
  int32_t nv;          // n (low 16 bits) | n_verify << 16, both unsigned 16-bit fields
  int32_t page_start;  // offset of the request's pages in page_indices
  int32_t item_start;  // first main-kernel work item
  int32_t part_start;  // first partial column in the workspace (split requests)
  int32_t comb_start;  // first combine work item (split requests)
};

// A request of a launch with overlap branches: its rows after the verify
// rows are branches, described by up to three words, each packed as rows
// (bits 0-15) | prefix verify rows kept (bits 16-27) | committed lead rows
// (bits 28-31), and `rep`: the word at index rep >> 28 stands for
// rep & 0xffff branches of its shape whose prefixes grow by
// (rep >> 16) & 0xfff each (a regular family, e.g. one draft block per
// hypothetical accepted length); the other words for one branch each.
// br[0] = 0 means no branch list (the rows after the verify rows are one
// continuation block that keeps every verify row).
struct AttnReqBr : AttnReq {
  int32_t br[3];
  int32_t rep;
};
constexpr int kMaxReqPerLaunchBr = 64;  // equals RG_BRANCH_MAX_REQS_PER_LAUNCH

template <typename Req, int MaxReq>
struct AttnPlanT {
  int32_t num_req;         // requests in this launch
  int32_t chunk;           // keys per work item, multiple of kKeyTile
  int32_t total_items;     // main-kernel work items
  int32_t total_comb;      // combine work items
  int32_t grid_items;      // total_items rounded up to a multiple of 8
  int32_t grid_comb;       // total_comb rounded up to a multiple of 8
  int32_t cols_per_group;  // query columns one work group covers (256)
  int32_t max_chunks;      // most chunks of one split request (picks the combine variant)
  int32_t persist_grid;    // 0: main kernel + combine kernel; else the work groups of the
                           // one-launch work-queue kernel (main items, then combine items)
  Req req[MaxReq + 1];     // entry num_req holds the end sentinels
};
using AttnPlan = AttnPlanT<AttnReq, kMaxReqPerLaunch>;
using AttnPlanBr = AttnPlanT<AttnReqBr, kMaxReqPerLaunchBr>;
static_assert(sizeof(AttnPlan) <= 3700, "attention plan must fit the kernel argument block");
static_assert(sizeof(AttnPlanBr) <= 3700, "attention plan must fit the kernel argument block");

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  uint16_t* out;
  float* lse;
  const int32_t* page_indices;
  uint16_t* part_o;  // per 32-column tile: 32 x D bf16 normalised partial outputs, MFMA fragment order
  float* part_ml;  // [partial columns][2] fp32 (running max of raw scores, sum)
  int32_t* sync;   // kSyncWords words, zero between calls: queue head, exit count, give-up
                   // flag, report word (nonzero after a call whose wait gave up, until
                   // read), then finished-tile counts (indexed by a column group's first
                   // combine item) and, kMaxSyncComb words on, started-combine counts
  int32_t hq, hkv, g;
  float sm_scale;    // natural-log domain scale
  float scale_log2;   // sm_scale * log2(e)
  float rescale_gap;  // raw-score margin before the running maximum moves
};

// Attention launchers (attention.hip).  `plan` is one launch's plan.
hipError_t launch_attention(const AttnArgs& args, const AttnPlan& plan, int head_dim,
                            hipStream_t stream);
hipError_t launch_attention(const AttnArgs& args, const AttnPlanBr& plan, int head_dim,
                            hipStream_t stream);

// Logit-row reductions (logits.hip).
constexpr int kLogitThreads = 256;
constexpr int kLogitChunk = 8192;  // vocab entries per work group

struct VerifyArgs {
  const uint16_t* logits;
  int64_t row_stride;
  int32_t vocab, num_req, rows, nchunk;
  int32_t cshift;      // row work groups are slots of 2^cshift >= nchunk chunks
  const int32_t* row_indptr;
  const int32_t* tokens;
  int32_t* row_argmax;
  int32_t* accept_len;
  int32_t* next_token;
  float* row_entropy;
  float* accept_entropy;
  float4* chunk_st;    // workspace [rows * nchunk] (max, bits(argmax), Z', S)
  int32_t vec;         // 16-byte loads allowed
  int32_t grid_rows;   // row work groups (rows << cshift rounded up to 8)
};

struct DraftArgs {
  const uint16_t* logits;
  int64_t row_stride;
  int32_t vocab, rows, nchunk;
  int32_t cshift;      // as in VerifyArgs
  int32_t* top1;
  int32_t* top2;
  float* p1;
  float* p2;
  float* margin;
  float* entropy;
  float4* chunk_a;       // workspace [rows * nchunk] (max, bits(i1), v2, bits(i2))
  float2* chunk_b;       // [rows * nchunk] (Z', S)
  int32_t vec;
  int32_t grid_rows;
};

inline int32_t logit_chunks(int32_t vocab) { return (vocab + kLogitChunk - 1) / kLogitChunk; }
// log2 of the chunk slots per row: the smallest power of two >= the row's
// chunks, so a row work group finds its row and chunk by shift and mask.
inline int32_t logit_chunk_shift(int32_t vocab) {
  int32_t s = 0;
  while ((1 << s) < logit_chunks(vocab)) ++s;
  return s;
}
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream);
hipError_t launch_draft(const DraftArgs& a, hipStream_t stream);
// Verify and draft passes of one round together: two launches in all.
hipError_t launch_round(const VerifyArgs& v, const DraftArgs& d, hipStream_t stream);

// Static device scratch of the allocation-free logit round (logits.hip):
// its size, and this device's address of it (looked up on first use).
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;  // equals RG_NOALLOC_SCRATCH_BYTES
hipError_t noalloc_scratch(void** ptr);

// Branch planning and matching (branches.hip).
struct PlanBranchArgs {
  const float* margin;
  const int32_t* top2;
  const int32_t* row_indptr;
  int32_t num_req;
  float delta;
  int32_t* n_risky;
  int32_t* n_corr;
  int32_t* corr_pos;
  int32_t* corr_tok;
  int32_t* continuation;
};
struct MatchBranchArgs {
  const int32_t* accept_len;
  const int32_t* next_token;
  const int32_t* block_len;
  const int32_t* n_corr;
  const int32_t* corr_pos;
  const int32_t* corr_tok;
  const int32_t* continuation;
  const int32_t* cont_first;
  int32_t num_req;
  int32_t* reused;
};
hipError_t launch_plan_branches(const PlanBranchArgs& a, hipStream_t stream);
hipError_t launch_match_branches(const MatchBranchArgs& a, hipStream_t stream);

// Verification-guided block sizing and bucketing (Sec. 5.2, Sec. 5.3).
constexpr int kMaxBlockCandidates = 8;
constexpr int kMaxSBins = 64;
constexpr int kMaxBucketRequests = 65536;
struct BlockSizeArgs {
  int32_t nb, ns;                       // candidates, s bins
  int32_t cand[kMaxBlockCandidates];    // ascending block sizes
  float edges[kMaxSBins - 1];           // ascending s-bin edges
  float cost[kMaxBlockCandidates];      // T_C(B)
  float rho;
  const float* value;                   // [nb][ns][nb][2]
  const int32_t* accept_len;
  const float* accept_entropy;
  const int32_t* prev_block;
  float* entropy_hist;
  int32_t num_req;
  int32_t* next_block;
  int32_t* order;                       // NULL when not grouping or when num_req == 0
  int32_t* bucket_offsets;              // NULL: no grouping
};
hipError_t launch_plan_block_sizes(const BlockSizeArgs& a, hipStream_t stream);

}  // namespace rg

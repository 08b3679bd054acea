// C ABI of the draft-verify hot path: argument validation, planning of the
// ragged attention batch, workspace carving and kernel launches.
//
// Planning reads only the host copies of the per-request sizes and turns
// them into launch arguments (AttnPlan): no table is uploaded and nothing is
// synchronised, so a call costs its kernel launches and nothing else on the
// stream.
#include "recguide.h"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "rg_internal.h"

static_assert(RG_BLOCK_MAX_CANDIDATES == rg::kMaxBlockCandidates, "header and kernel limits agree");
static_assert(RG_BLOCK_MAX_S_BINS == rg::kMaxSBins, "header and kernel limits agree");
static_assert(RG_BLOCK_MAX_REQUESTS == rg::kMaxBucketRequests, "header and kernel limits agree");
static_assert(RG_BRANCH_MAX_REQS_PER_LAUNCH == rg::kMaxReqPerLaunchBr, "header and kernel limits agree");
static_assert(RG_NOALLOC_SCRATCH_BYTES == rg::kNoAllocScratchBytes, "header and scratch size agree");

namespace {

using namespace rg;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

int env_int(const char* name, int fallback) {
  const char* v = std::getenv(name);
  if (v == nullptr || *v == 0) return fallback;
  return std::atoi(v);
}

rg_status validate_layout(const rg_attn_layout* L) {
  if (L == nullptr) return RG_ERR_NULL;
  if (!L->q_indptr || !L->n_verify || !L->ctx_len || !L->page_indptr || !L->page_indices) return RG_ERR_NULL;
  if (L->num_requests < 1 || L->num_q_heads < 1 || L->num_kv_heads < 1 || L->num_pages < 1) return RG_ERR_SHAPE;
  if (L->num_q_heads % L->num_kv_heads != 0) return RG_ERR_SHAPE;
  if (L->head_dim != 64 && L->head_dim != 128) return RG_ERR_UNSUPPORTED;
  if (L->page_size != kPageSize) return RG_ERR_UNSUPPORTED;
  if (L->q_indptr[0] != 0 || L->page_indptr[0] != 0) return RG_ERR_SHAPE;
  for (int r = 0; r < L->num_requests; ++r) {
    const int64_t n = (int64_t)L->q_indptr[r + 1] - L->q_indptr[r];
    const int64_t pages = (int64_t)L->page_indptr[r + 1] - L->page_indptr[r];
    if (n < 0 || pages < 0 || L->ctx_len[r] < 0) return RG_ERR_SHAPE;
    if (L->n_verify[r] < 0 || L->n_verify[r] > n) return RG_ERR_SHAPE;
    if (n > 0xffff) return RG_ERR_UNSUPPORTED;  // query rows per request
    const int64_t T = (int64_t)L->ctx_len[r] + n;
    if (T > (int64_t(1) << 30)) return RG_ERR_UNSUPPORTED;
    if (n > 0 && pages * kPageSize < T) return RG_ERR_SHAPE;
  }
  return RG_OK;
}

// Branch layout of the overlap (Sec. 5.1): at most three branches per
// request, each within its packing limits, and a listed set of branches
// covers exactly the request's rows after its verify rows.
// Packs request r's branch list into at most three words plus a repeat
// word: the longest trailing run of branches with equal rows and lead whose
// prefixes grow by a constant step >= 0 becomes one word standing for
// `count` branches; the branches before it keep a word each.  False when
// more than two branches precede that run or the run exceeds the packing
// limits.
bool pack_branches(const rg_branch_layout* B, int r, int32_t (&w)[3], int32_t& rep) {
  w[0] = w[1] = w[2] = 0;
  rep = 0;
  if (B == nullptr) return true;
  const int k0 = B->branch_indptr[r], m = B->branch_indptr[r + 1] - k0;
  if (m == 0) return true;
  auto same = [&](int a, int b) { return B->rows[k0 + a] == B->rows[k0 + b] && B->lead[k0 + a] == B->lead[k0 + b]; };
  int j = m - 1, step = 0;
  if (m >= 2 && same(m - 1, m - 2) && B->prefix[k0 + m - 1] >= B->prefix[k0 + m - 2]) {
    step = B->prefix[k0 + m - 1] - B->prefix[k0 + m - 2];
    j = m - 2;
    while (j > 0 && same(j - 1, j) && B->prefix[k0 + j] - B->prefix[k0 + j - 1] == step) --j;
  }
  const int count = m - j;
  if (j > 2 || count > 0xffff || step > 0xfff) return false;
  for (int i = 0; i <= j; ++i) {
    const int k = k0 + i;
    w[i] = (int32_t)((uint32_t)B->rows[k] | ((uint32_t)B->prefix[k] << 16) | ((uint32_t)B->lead[k] << 28));
  }
  rep = (int32_t)((uint32_t)count | ((uint32_t)step << 16) | ((uint32_t)j << 28));
  return true;
}

rg_status validate_branches(const rg_attn_layout* L, const rg_branch_layout* B) {
  if (B == nullptr || !B->branch_indptr) return RG_ERR_NULL;
  if (B->branch_indptr[0] != 0) return RG_ERR_SHAPE;
  const int nb_all = B->branch_indptr[L->num_requests];
  if (nb_all > 0 && (!B->prefix || !B->lead || !B->rows)) return RG_ERR_NULL;
  for (int r = 0; r < L->num_requests; ++r) {
    const int nb = B->branch_indptr[r + 1] - B->branch_indptr[r];
    if (nb < 0) return RG_ERR_SHAPE;
    if (nb == 0) continue;
    const int64_t n = (int64_t)L->q_indptr[r + 1] - L->q_indptr[r];
    const int V = L->n_verify[r];
    int64_t sum = 0;
    for (int k = B->branch_indptr[r]; k < B->branch_indptr[r + 1]; ++k) {
      if (B->rows[k] < 1 || B->prefix[k] < 0 || B->prefix[k] > V || B->lead[k] < 0 || B->lead[k] > B->rows[k])
        return RG_ERR_SHAPE;
      if (B->rows[k] > 0xffff || B->prefix[k] > 0xfff || B->lead[k] > 0xf) return RG_ERR_UNSUPPORTED;
      sum += B->rows[k];
    }
    if (sum != n - V) return RG_ERR_SHAPE;
    int32_t w[3], rep;
    if (!pack_branches(B, r, w, rep)) return RG_ERR_UNSUPPORTED;
  }
  return RG_OK;
}

template <typename Plan>
struct FullPlanT {
  std::vector<Plan> launches;
  int chunk = 0;
  int cols_per_group = 256;
  int64_t items = 0, split_requests = 0, max_partial_cols = 0, total_partial_cols = 0;
  int64_t max_comb = 0;
  int persistent_launches = 0;
  size_t ws_bytes = 0;
  size_t o_offset = 0;
  size_t ml_offset = 0;
  size_t sync_offset = 0;
};

// Compute units of the current device: the rounds of the chunk rule and the
// one-launch kernel's work groups (one per CU); 256 (MI355X) when the runtime
// cannot say.  Every planning call (workspace query, plan query, the call
// itself) asks, so on one device they all plan alike.
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return n;
}

// Keys per work item.  An item costs a fixed start-up and wind-down (request
// lookup, page numbers, first copies, epilogue: several microseconds) besides
// its keys, and splitting a request adds partial outputs and the combine
// kernel; items are dispatched costliest request first, and one work group
// fills a CU, so items run in rounds of `num_cus` (256 on MI355X).  The rule:
// the shortest chunk (a multiple of the LDS buffer, at least 256 keys, at most
// S = all keys / num_cus, one CU's share) whose items fit in two rounds -- the finest split that
// leaves no third round for a few items to run alone; when even chunks of S
// give more than two rounds, chunks of S (requests no longer than S stay
// whole).  `pair_keys` holds T of every (request, column group); each stands
// for Hkv pairs, one per KV head.  Measured on twelve `mid` draws against
// the earlier rule (the longest chunk still giving two items per CU, which
// usually left a short third round): -9.2 % on average, from 0 to -15 %
// (same-host A/B); `tiny`, `low`, `high` and `long` get the same chunks as
// before.  Earlier
// measurements behind the bounds: uneven splits hurt most (at `long`,
// 24576-key chunks, a full chunk plus a short remainder per request, took
// 1633 us against 1340 us whole), and finer chunks cost more than a dispatch
// model with a fixed start-up predicts (merge work, partial traffic).
int choose_chunk(const std::vector<int64_t>& pair_keys, int hkv, int num_cus) {
  const int forced = env_int("RG_ATTN_CHUNK", 0);
  if (forced > 0) return (int)std::min<int64_t>(kMaxChunkKeys, round_up(forced, kKeyTile));
  const int64_t kCUs = std::max(1, num_cus);
  const int64_t kTwoRounds = 2 * kCUs;
  const int64_t floor_keys = round_up(std::max(kKeyTile, env_int("RG_ATTN_MIN_CHUNK", 256)), kKeyTile);
  int64_t total = 0, longest = 0;
  for (int64_t t : pair_keys) {
    total += t * hkv;
    longest = std::max(longest, t);
  }
  const int64_t share = total / kCUs;
  const int64_t whole = std::min<int64_t>(kMaxChunkKeys, std::max(floor_keys, round_up(longest, kKeyTile)));
  auto items = [&](int64_t chunk) {  // nonincreasing in chunk
    int64_t n = 0;
    for (int64_t t : pair_keys) n += (t + chunk - 1) / chunk;
    return n * hkv;
  };
  const int64_t hi_keys = std::min(whole, std::max(floor_keys, round_up(share, kKeyTile)));
  if (items(hi_keys) > kTwoRounds) return (int)hi_keys;
  if (items(floor_keys) <= kTwoRounds) return (int)floor_keys;
  // Buffers per chunk: items(lo) > two rounds >= items(hi).
  int64_t lo = floor_keys / kKeyTile, hi = hi_keys / kKeyTile;
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) / 2;
    if (items(mid * kKeyTile) <= kTwoRounds) hi = mid;
    else lo = mid;
  }
  return (int)(hi * kKeyTile);
}

// Branch words of request r (see AttnReqBr); all zero when B is NULL or
// the request lists no branch.

// Launches with a split request run as the main kernel plus the combine
// kernel, or, with RG_ATTN_PERSIST=1, as one work-queue launch (main items,
// then the combine items; `num_cus` work groups at most).  The two launches
// are the default because they measured faster on MI355X at every workload:
// the device-scope counting and waiting that replaces the kernel boundary
// costs about as much as the boundary itself.
template <typename Plan, int MaxReq>
rg_status plan_attention(const rg_attn_layout* L, const rg_branch_layout* B, FullPlanT<Plan>& fp,
                         int num_cus) {
  const int R = L->num_requests;
  const bool persist = env_int("RG_ATTN_PERSIST", 0) != 0;
  // 16-byte rows per combine item: 128 (combine kernel), 256 (one-launch kernel)
  const int comb_rows = persist ? 256 : 128;
  const int g = L->num_q_heads / L->num_kv_heads;
  const int hkv = L->num_kv_heads;
  fp.cols_per_group = 256;  // 8 waves x 32 columns per work group
  std::vector<int64_t> pair_keys;  // one entry per (request, column group): Hkv pairs each
  for (int r = 0; r < R; ++r) {
    const int64_t n = L->q_indptr[r + 1] - L->q_indptr[r];
    if (n == 0) continue;
    const int64_t ncg = (n * g + fp.cols_per_group - 1) / fp.cols_per_group;
    for (int64_t cg = 0; cg < ncg; ++cg) pair_keys.push_back((int64_t)L->ctx_len[r] + n);
  }
  fp.chunk = choose_chunk(pair_keys, hkv, num_cus);
  // Costliest work items first: work groups are dispatched in item order, so
  // the long items start early and the short ones fill in at the end.  An
  // item's time is estimated in units of one 128-key buffer at the copy rate:
  // about two units of start-up plus its buffers, each costing
  // max(1, tiles / 4) units for its 32-column tiles -- wide items are bound
  // by their MFMA and softmax work, not by the copies.  A request's items all
  // get the estimate of its widest column group's full-chunk item.  The
  // divisor was picked by measurement: against ordering by keys alone, over 4
  // `long` and 10 `mid` draws, the divisors 4 and 5.6 and a linear
  // 1 + tiles / 8 gave `long` -3.1, -0.8 and -3.5 %, `mid` -1.6, -1.8 and
  // -1.2 %, and `high` (narrow items) +0.2, +0.2 and +0.7 %.
  std::vector<double> cost(R);
  for (int r = 0; r < R; ++r) {
    const int64_t n = L->q_indptr[r + 1] - L->q_indptr[r];
    const int64_t T = (int64_t)L->ctx_len[r] + n;
    const int64_t all_tiles = (n * g + 31) / 32;
    const int64_t groups = std::max<int64_t>(1, (all_tiles + 7) / 8);
    const int64_t tiles = (all_tiles + groups - 1) / groups;  // the widest column group's (tiles dealt evenly)
    const int64_t bufs = (std::min<int64_t>(T, fp.chunk) + kKeyTile - 1) / kKeyTile;
    cost[r] = n == 0 ? 0.0 : 2.0 + (double)bufs * std::max(1.0, (double)tiles / 4.0);
  }
  std::vector<int> order(R);
  for (int r = 0; r < R; ++r) order[r] = r;
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
    if (cost[x] != cost[y]) return cost[x] > cost[y];
    return (int64_t)L->ctx_len[x] + (L->q_indptr[x + 1] - L->q_indptr[x]) >
           (int64_t)L->ctx_len[y] + (L->q_indptr[y + 1] - L->q_indptr[y]);
  });
  for (int r0 = 0; r0 < R; r0 += MaxReq) {
    const int cnt = std::min(MaxReq, R - r0);
    Plan p;
    std::memset(&p, 0, sizeof(p));
    p.num_req = cnt;
    p.chunk = fp.chunk;
    p.cols_per_group = fp.cols_per_group;
    int64_t items = 0, part = 0, comb = 0;
    for (int k = 0; k < cnt; ++k) {
      const int r = order[r0 + k];
      const int64_t n = L->q_indptr[r + 1] - L->q_indptr[r];
      auto& q = p.req[k];
      if constexpr (__is_same(Plan, AttnPlanBr)) pack_branches(B, r, q.br, q.rep);
      q.q_start = L->q_indptr[r];
      q.ctx = L->ctx_len[r];
      q.nv = (int32_t)(n | ((int64_t)L->n_verify[r] << 16));
      q.page_start = L->page_indptr[r];
      q.item_start = (int32_t)items;
      q.part_start = (int32_t)part;
      q.comb_start = (int32_t)comb;
      if (n == 0) continue;
      const int64_t M = n * g;
      const int64_t T = (int64_t)L->ctx_len[r] + n;
      const int64_t nch = (T + fp.chunk - 1) / fp.chunk;
      const int64_t ncg = (M + fp.cols_per_group - 1) / fp.cols_per_group;
      items += hkv * ncg * nch;
      if (nch > 1) {
        p.max_chunks = std::max<int32_t>(p.max_chunks, (int32_t)nch);
        // partials are stored per 32-column tile, so columns round up to 32
        part += hkv * nch * round_up(M, 32);
        comb += hkv * ((M + 31) / 32) * (L->head_dim * 4 / comb_rows);  // slices of a tile's 4 D rows
        fp.split_requests += 1;
      }
      if (items > INT32_MAX / 2 || part > INT32_MAX / 2) return RG_ERR_UNSUPPORTED;
    }
    p.req[cnt].item_start = (int32_t)items;
    p.req[cnt].part_start = (int32_t)part;
    p.req[cnt].comb_start = (int32_t)comb;
    p.total_items = (int32_t)items;
    p.total_comb = (int32_t)comb;
    p.grid_items = (int32_t)round_up(items, 8);
    p.grid_comb = (int32_t)round_up(comb, 8);
    if (persist && comb > 0 && comb <= kMaxSyncComb) {
      p.persist_grid = (int32_t)round_up(std::min<int64_t>(items + comb, std::max(8, num_cus)), 8);
      fp.persistent_launches += 1;
    }
    fp.items += items;
    fp.max_partial_cols = std::max(fp.max_partial_cols, part);
    fp.total_partial_cols += part;
    fp.max_comb = std::max(fp.max_comb, comb);
    fp.launches.push_back(p);
  }
  // Workspace: the one-launch kernel's synchronisation words first, at a
  // fixed place and size (zero before the first call; every call leaves them
  // zero, whatever its layout), then the partial outputs and their (max, sum).
  const size_t sync_bytes = align256((size_t)kSyncWords * sizeof(int32_t));
  const size_t o_bytes = align256((size_t)fp.max_partial_cols * L->head_dim * sizeof(uint16_t));
  const size_t ml_bytes = align256((size_t)fp.max_partial_cols * 2 * sizeof(float));
  fp.sync_offset = 0;
  fp.o_offset = sync_bytes;
  fp.ml_offset = sync_bytes + o_bytes;
  fp.ws_bytes = fp.max_partial_cols ? sync_bytes + o_bytes + ml_bytes : 0;
  return RG_OK;
}

size_t verify_ws_bytes(int32_t rows, int32_t vocab) {
  return align256((size_t)rows * logit_chunks(vocab) * 16);
}

size_t draft_ws_bytes(int32_t rows, int32_t vocab) {
  const size_t nchunk = logit_chunks(vocab);
  return align256((size_t)rows * nchunk * 16) + align256((size_t)rows * nchunk * 8);
}

}  // namespace

extern "C" {

int32_t rg_abi_version(void) { return RG_ABI_VERSION; }

const char* rg_status_string(rg_status s) {
  switch (s) {
    case RG_OK: return "ok";
    case RG_ERR_NULL: return "a required pointer is NULL";
    case RG_ERR_SHAPE: return "inconsistent sizes or offsets";
    case RG_ERR_UNSUPPORTED: return "unsupported configuration";
    case RG_ERR_WORKSPACE: return "workspace missing or too small";
    case RG_ERR_HIP: return "HIP launch or runtime error";
    case RG_ERR_WAIT: return "a one-launch attention wait gave up";
    default: return "unknown status";
  }
}

}  // extern "C"

namespace {

using FullPlan = FullPlanT<AttnPlan>;
using FullPlanBr = FullPlanT<AttnPlanBr>;

rg_status plan_plain(const rg_attn_layout* layout, FullPlan& fp, int num_cus) {
  return plan_attention<AttnPlan, kMaxReqPerLaunch>(layout, nullptr, fp, num_cus);
}
rg_status plan_branched(const rg_attn_layout* layout, const rg_branch_layout* branches, FullPlanBr& fp,
                        int num_cus) {
  rg_status st = validate_branches(layout, branches);
  if (st != RG_OK) return st;
  return plan_attention<AttnPlanBr, kMaxReqPerLaunchBr>(layout, branches, fp, num_cus);
}

template <typename Plan>
rg_status run_attention(const rg_attn_layout* layout, const FullPlanT<Plan>& fp, const uint16_t* q,
                        const uint16_t* k_cache, const uint16_t* v_cache, uint16_t* out, float* lse,
                        void* ws, size_t ws_bytes, void* stream) {
  if (!q || !k_cache || !v_cache || !out) return RG_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
      (lse && !aligned(lse, 4)) || !aligned(layout->page_indices, 4))
    return RG_ERR_UNSUPPORTED;
  if (fp.ws_bytes > 0 && (ws == nullptr || ws_bytes < fp.ws_bytes || !aligned(ws, 16))) return RG_ERR_WORKSPACE;

  AttnArgs a;
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.out = out;
  a.lse = lse;
  a.page_indices = layout->page_indices;
  a.part_o = fp.ws_bytes ? reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + fp.o_offset) : nullptr;
  a.part_ml = fp.ws_bytes ? reinterpret_cast<float*>(static_cast<char*>(ws) + fp.ml_offset) : nullptr;
  a.sync = fp.ws_bytes ? reinterpret_cast<int32_t*>(static_cast<char*>(ws) + fp.sync_offset) : nullptr;
  a.hq = layout->num_q_heads;
  a.hkv = layout->num_kv_heads;
  a.g = layout->num_q_heads / layout->num_kv_heads;
  a.sm_scale = layout->sm_scale > 0.f ? layout->sm_scale : 1.0f / std::sqrt((float)layout->head_dim);
  a.scale_log2 = a.sm_scale * 1.4426950408889634f;
  a.rescale_gap = 8.0f / a.scale_log2;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (const Plan& p : fp.launches) {
    if (p.total_items == 0) continue;
    if (launch_attention(a, p, layout->head_dim, s) != hipSuccess) return RG_ERR_HIP;
  }
  return RG_OK;
}

}  // namespace

extern "C" {

rg_status rg_draft_verify_attention_workspace(const rg_attn_layout* layout, size_t* bytes) {
  if (bytes == nullptr) return RG_ERR_NULL;
  rg_status st = validate_layout(layout);
  if (st != RG_OK) return st;
  FullPlan fp;
  st = plan_plain(layout, fp, device_cus());
  if (st != RG_OK) return st;
  *bytes = fp.ws_bytes;
  return RG_OK;
}

rg_status rg_draft_verify_attention_check(void* ws, size_t ws_bytes, void* stream) {
  if (ws == nullptr) return RG_ERR_NULL;
  if (ws_bytes < (size_t)kSyncHeader * sizeof(int32_t)) return RG_ERR_WORKSPACE;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return RG_ERR_HIP;
  int32_t* report = static_cast<int32_t*>(ws) + 3;  // sync word 3, at the workspace's start
  int32_t word = 0;
  if (hipMemcpy(&word, report, sizeof(word), hipMemcpyDeviceToHost) != hipSuccess) return RG_ERR_HIP;
  if (word == 0) return RG_OK;
  const int32_t zero = 0;
  if (hipMemcpy(report, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return RG_ERR_HIP;
  return RG_ERR_WAIT;
}

rg_status rg_draft_verify_attention_plan(const rg_attn_layout* layout, rg_attn_plan_info* info) {
  if (info == nullptr) return RG_ERR_NULL;
  rg_status st = validate_layout(layout);
  if (st != RG_OK) return st;
  FullPlan fp;
  st = plan_plain(layout, fp, device_cus());
  if (st != RG_OK) return st;
  info->num_launches = (int32_t)fp.launches.size();
  info->chunk_keys = fp.chunk;
  info->work_items = fp.items;
  info->split_requests = fp.split_requests;
  info->partial_columns = fp.total_partial_cols;
  info->workspace_bytes = (int64_t)fp.ws_bytes;
  info->persistent_launches = fp.persistent_launches;
  info->sync_words = fp.ws_bytes ? kSyncWords : 0;
  info->sync_offset = fp.ws_bytes ? (int64_t)fp.sync_offset : -1;
  return RG_OK;
}

rg_status rg_draft_verify_attention(const rg_attn_layout* layout, const uint16_t* q,
                                    const uint16_t* k_cache, const uint16_t* v_cache,
                                    uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                                    void* stream) {
  rg_status st = validate_layout(layout);
  if (st != RG_OK) return st;
  FullPlan fp;
  st = plan_plain(layout, fp, device_cus());
  if (st != RG_OK) return st;
  return run_attention(layout, fp, q, k_cache, v_cache, out, lse, ws, ws_bytes, stream);
}

rg_status rg_multibranch_attention_workspace(const rg_attn_layout* layout, const rg_branch_layout* branches,
                                             size_t* bytes) {
  if (bytes == nullptr) return RG_ERR_NULL;
  rg_status st = validate_layout(layout);
  if (st != RG_OK) return st;
  FullPlanBr fp;
  st = plan_branched(layout, branches, fp, device_cus());
  if (st != RG_OK) return st;
  *bytes = fp.ws_bytes;
  return RG_OK;
}

rg_status rg_multibranch_attention(const rg_attn_layout* layout, const rg_branch_layout* branches,
                                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                   uint16_t* out, float* lse, void* ws, size_t ws_bytes, void* stream) {
  rg_status st = validate_layout(layout);
  if (st != RG_OK) return st;
  FullPlanBr fp;
  st = plan_branched(layout, branches, fp, device_cus());
  if (st != RG_OK) return st;
  return run_attention(layout, fp, q, k_cache, v_cache, out, lse, ws, ws_bytes, stream);
}

rg_status rg_verify_accept_workspace(int32_t num_requests, int32_t total_rows, int32_t vocab, size_t* bytes) {
  if (bytes == nullptr) return RG_ERR_NULL;
  if (num_requests < 1 || total_rows < 0 || vocab < 1) return RG_ERR_SHAPE;
  *bytes = verify_ws_bytes(total_rows, vocab);
  return RG_OK;
}

}  // extern "C"

namespace {

rg_status make_verify_args(const uint16_t* logits, int64_t row_stride, int32_t vocab, int32_t num_requests,
                           int32_t total_rows, const int32_t* row_indptr, const int32_t* draft_tokens,
                           int32_t* row_argmax, int32_t* accept_len, int32_t* next_token, float* row_entropy,
                           float* accept_entropy, void* ws, size_t ws_bytes, VerifyArgs& a) {
  if (num_requests < 1 || total_rows < 0 || vocab < 1) return RG_ERR_SHAPE;
  if (!row_indptr || !accept_len || !next_token) return RG_ERR_NULL;
  if (total_rows > 0 && (!logits || !draft_tokens || !row_argmax)) return RG_ERR_NULL;
  if (row_stride < vocab) return RG_ERR_SHAPE;
  if (((int64_t)total_rows << logit_chunk_shift(vocab)) > INT32_MAX / 2) return RG_ERR_UNSUPPORTED;
  const size_t need = verify_ws_bytes(total_rows, vocab);
  if (total_rows > 0 && (ws == nullptr || ws_bytes < need || !aligned(ws, 16))) return RG_ERR_WORKSPACE;
  std::memset(&a, 0, sizeof(a));
  a.logits = logits;
  a.row_stride = row_stride;
  a.vocab = vocab;
  a.num_req = num_requests;
  a.rows = total_rows;
  a.nchunk = logit_chunks(vocab);
  a.cshift = logit_chunk_shift(vocab);
  a.row_indptr = row_indptr;
  a.tokens = draft_tokens;
  a.row_argmax = row_argmax;
  a.accept_len = accept_len;
  a.next_token = next_token;
  a.row_entropy = row_entropy;
  a.accept_entropy = accept_entropy;
  a.chunk_st = static_cast<float4*>(ws);
  a.vec = (aligned(logits, 16) && row_stride % 8 == 0) ? 1 : 0;
  a.grid_rows = (int32_t)round_up((int64_t)total_rows << a.cshift, 8);
  return RG_OK;
}

rg_status make_draft_args(const uint16_t* logits, int64_t row_stride, int32_t vocab, int32_t total_rows,
                          int32_t* top1, int32_t* top2, float* p1, float* p2, float* margin, float* entropy,
                          void* ws, size_t ws_bytes, DraftArgs& a) {
  if (total_rows < 0 || vocab < 2) return RG_ERR_SHAPE;
  if (total_rows > 0 && (!logits || !top1 || !top2 || !p1 || !p2)) return RG_ERR_NULL;
  if (row_stride < vocab) return RG_ERR_SHAPE;
  if (((int64_t)total_rows << logit_chunk_shift(vocab)) > INT32_MAX / 2) return RG_ERR_UNSUPPORTED;
  const size_t need = draft_ws_bytes(total_rows, vocab);
  if (total_rows > 0 && (ws == nullptr || ws_bytes < need || !aligned(ws, 16))) return RG_ERR_WORKSPACE;
  std::memset(&a, 0, sizeof(a));
  a.logits = logits;
  a.row_stride = row_stride;
  a.vocab = vocab;
  a.rows = total_rows;
  a.nchunk = logit_chunks(vocab);
  a.cshift = logit_chunk_shift(vocab);
  a.top1 = top1;
  a.top2 = top2;
  a.p1 = p1;
  a.p2 = p2;
  a.margin = margin;
  a.entropy = entropy;
  char* w = static_cast<char*>(ws);
  a.chunk_a = reinterpret_cast<float4*>(w);
  if (w != nullptr) w += align256((size_t)total_rows * a.nchunk * 16);
  a.chunk_b = reinterpret_cast<float2*>(w);
  a.vec = (aligned(logits, 16) && row_stride % 8 == 0) ? 1 : 0;
  a.grid_rows = (int32_t)round_up((int64_t)total_rows << a.cshift, 8);
  return RG_OK;
}

}  // namespace

extern "C" {

rg_status rg_verify_accept(const uint16_t* logits, int64_t row_stride, int32_t vocab,
                           int32_t num_requests, int32_t total_rows, const int32_t* row_indptr,
                           const int32_t* draft_tokens, int32_t* row_argmax, int32_t* accept_len,
                           int32_t* next_token, float* row_entropy, float* accept_entropy,
                           void* ws, size_t ws_bytes, void* stream) {
  VerifyArgs a;
  const rg_status st = make_verify_args(logits, row_stride, vocab, num_requests, total_rows, row_indptr,
                                        draft_tokens, row_argmax, accept_len, next_token, row_entropy,
                                        accept_entropy, ws, ws_bytes, a);
  if (st != RG_OK) return st;
  return launch_verify(a, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

rg_status rg_draft_confidence_workspace(int32_t total_rows, int32_t vocab, size_t* bytes) {
  if (bytes == nullptr) return RG_ERR_NULL;
  if (total_rows < 0 || vocab < 2) return RG_ERR_SHAPE;
  *bytes = draft_ws_bytes(total_rows, vocab);
  return RG_OK;
}

rg_status rg_draft_confidence(const uint16_t* logits, int64_t row_stride, int32_t vocab,
                              int32_t total_rows, int32_t* top1, int32_t* top2, float* p1,
                              float* p2, float* margin, float* entropy, void* ws,
                              size_t ws_bytes, void* stream) {
  DraftArgs a;
  const rg_status st = make_draft_args(logits, row_stride, vocab, total_rows, top1, top2, p1, p2, margin,
                                       entropy, ws, ws_bytes, a);
  if (st != RG_OK) return st;
  if (total_rows == 0) return RG_OK;
  return launch_draft(a, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

rg_status rg_verify_and_confidence_workspace(int32_t num_requests, int32_t verify_rows, int32_t draft_rows,
                                             int32_t vocab, size_t* bytes) {
  if (bytes == nullptr) return RG_ERR_NULL;
  if (num_requests < 1 || verify_rows < 0 || draft_rows < 0 || vocab < 2) return RG_ERR_SHAPE;
  *bytes = align256(verify_ws_bytes(verify_rows, vocab)) + draft_ws_bytes(draft_rows, vocab);
  return RG_OK;
}

rg_status rg_verify_and_confidence(const uint16_t* verify_logits, int64_t verify_stride,
                                   const uint16_t* draft_logits, int64_t draft_stride, int32_t vocab,
                                   int32_t num_requests, int32_t verify_rows, const int32_t* row_indptr,
                                   const int32_t* draft_tokens, int32_t* row_argmax, int32_t* accept_len,
                                   int32_t* next_token, float* row_entropy, float* accept_entropy,
                                   int32_t draft_rows, int32_t* top1, int32_t* top2, float* p1, float* p2,
                                   float* margin, float* entropy, void* ws, size_t ws_bytes, void* stream) {
  if (vocab < 2 || verify_rows < 0 || draft_rows < 0) return RG_ERR_SHAPE;
  const size_t vbytes = align256(verify_ws_bytes(verify_rows, vocab));
  const size_t dbytes = draft_ws_bytes(draft_rows, vocab);
  if (vbytes + dbytes > 0 && (ws == nullptr || ws_bytes < vbytes + dbytes || !aligned(ws, 256)))
    return RG_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  VerifyArgs v;
  rg_status st = make_verify_args(verify_logits, verify_stride, vocab, num_requests, verify_rows, row_indptr,
                                  draft_tokens, row_argmax, accept_len, next_token, row_entropy, accept_entropy,
                                  w, vbytes, v);
  if (st != RG_OK) return st;
  DraftArgs d;
  st = make_draft_args(draft_logits, draft_stride, vocab, draft_rows, top1, top2, p1, p2, margin, entropy,
                       dbytes ? w + vbytes : nullptr, dbytes, d);
  if (st != RG_OK) return st;
  return launch_round(v, d, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

rg_status rg_verify_and_confidence_noalloc(const uint16_t* verify_logits, int64_t verify_stride,
                                           const uint16_t* draft_logits, int64_t draft_stride, int32_t vocab,
                                           int32_t num_requests, int32_t verify_rows, const int32_t* row_indptr,
                                           const int32_t* draft_tokens, int32_t* row_argmax, int32_t* accept_len,
                                           int32_t* next_token, float* row_entropy, float* accept_entropy,
                                           int32_t draft_rows, int32_t* top1, int32_t* top2, float* p1, float* p2,
                                           float* margin, float* entropy, void* stream) {
  // The same workspace layout as rg_verify_and_confidence, carved from the
  // static scratch: sizes past it are refused before anything is looked up.
  size_t need = 0;
  const rg_status st = rg_verify_and_confidence_workspace(num_requests, verify_rows, draft_rows, vocab, &need);
  if (st != RG_OK) return st;
  if (need > kNoAllocScratchBytes) return RG_ERR_UNSUPPORTED;
  void* ws = nullptr;
  if (need > 0 && noalloc_scratch(&ws) != hipSuccess) return RG_ERR_HIP;
  return rg_verify_and_confidence(verify_logits, verify_stride, draft_logits, draft_stride, vocab, num_requests,
                                  verify_rows, row_indptr, draft_tokens, row_argmax, accept_len, next_token,
                                  row_entropy, accept_entropy, draft_rows, top1, top2, p1, p2, margin, entropy,
                                  ws, need, stream);
}

rg_status rg_plan_branches(const float* margin, const int32_t* top2, const int32_t* row_indptr,
                           int32_t num_requests, int32_t total_rows, float delta, int32_t* n_risky,
                           int32_t* n_corr, int32_t* corr_pos, int32_t* corr_tok, int32_t* continuation,
                           void* stream) {
  if (num_requests < 1 || total_rows < 0) return RG_ERR_SHAPE;
  if (!row_indptr || !n_risky || !n_corr || !corr_pos || !corr_tok || !continuation) return RG_ERR_NULL;
  if (total_rows > 0 && (!margin || !top2)) return RG_ERR_NULL;
  PlanBranchArgs a;
  a.margin = margin;
  a.top2 = top2;
  a.row_indptr = row_indptr;
  a.num_req = num_requests;
  a.delta = delta;
  a.n_risky = n_risky;
  a.n_corr = n_corr;
  a.corr_pos = corr_pos;
  a.corr_tok = corr_tok;
  a.continuation = continuation;
  return launch_plan_branches(a, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

rg_status rg_match_branches(const int32_t* accept_len, const int32_t* next_token, const int32_t* block_len,
                            const int32_t* n_corr, const int32_t* corr_pos, const int32_t* corr_tok,
                            const int32_t* continuation, const int32_t* cont_first, int32_t num_requests,
                            int32_t* reused, void* stream) {
  if (num_requests < 1) return RG_ERR_SHAPE;
  if (!accept_len || !next_token || !block_len || !n_corr || !corr_pos || !corr_tok || !continuation ||
      !cont_first || !reused)
    return RG_ERR_NULL;
  MatchBranchArgs a;
  a.accept_len = accept_len;
  a.next_token = next_token;
  a.block_len = block_len;
  a.n_corr = n_corr;
  a.corr_pos = corr_pos;
  a.corr_tok = corr_tok;
  a.continuation = continuation;
  a.cont_first = cont_first;
  a.num_req = num_requests;
  a.reused = reused;
  return launch_match_branches(a, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

rg_status rg_plan_block_sizes(const rg_block_policy* policy, const int32_t* accept_len,
                              const float* accept_entropy, const int32_t* prev_block, float* entropy_hist,
                              int32_t num_requests, int32_t* next_block, int32_t* order,
                              int32_t* bucket_offsets, void* stream) {
  if (!policy) return RG_ERR_NULL;
  const int nb = policy->num_candidates, ns = policy->num_s_bins;
  if (nb < 1 || nb > kMaxBlockCandidates || ns < 1 || ns > kMaxSBins) return RG_ERR_UNSUPPORTED;
  if (!policy->candidates || !policy->cost || !policy->value || (ns > 1 && !policy->s_edges)) return RG_ERR_NULL;
  for (int i = 0; i < nb; ++i) {
    if (policy->candidates[i] < 1) return RG_ERR_SHAPE;
    if (i > 0 && policy->candidates[i] <= policy->candidates[i - 1]) return RG_ERR_SHAPE;
  }
  for (int i = 1; i + 1 < ns; ++i)
    if (!(policy->s_edges[i] >= policy->s_edges[i - 1])) return RG_ERR_SHAPE;
  if (num_requests < 0) return RG_ERR_SHAPE;
  if (num_requests > kMaxBucketRequests) return RG_ERR_UNSUPPORTED;
  // grouping is asked for by bucket_offsets; order may be NULL only when there is nothing to order
  if (order != nullptr && bucket_offsets == nullptr) return RG_ERR_NULL;
  if (bucket_offsets != nullptr && order == nullptr && num_requests > 0) return RG_ERR_NULL;
  if (num_requests > 0 && (!accept_len || !accept_entropy || !prev_block || !entropy_hist || !next_block))
    return RG_ERR_NULL;
  BlockSizeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.nb = nb;
  a.ns = ns;
  for (int i = 0; i < nb; ++i) {
    a.cand[i] = policy->candidates[i];
    a.cost[i] = policy->cost[i];
  }
  for (int i = 0; i + 1 < ns; ++i) a.edges[i] = policy->s_edges[i];
  a.rho = policy->rho;
  a.value = policy->value;
  a.accept_len = accept_len;
  a.accept_entropy = accept_entropy;
  a.prev_block = prev_block;
  a.entropy_hist = entropy_hist;
  a.num_req = num_requests;
  a.next_block = next_block;
  a.order = order;
  a.bucket_offsets = bucket_offsets;
  if (num_requests == 0 && bucket_offsets == nullptr) return RG_OK;
  return launch_plan_block_sizes(a, static_cast<hipStream_t>(stream)) == hipSuccess ? RG_OK : RG_ERR_HIP;
}

}  // extern "C"

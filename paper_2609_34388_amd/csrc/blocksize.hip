// Verification-guided block sizing (Sec. 5.2, Eq. 2 and 3) and block-size
// bucketing (Sec. 5.3), gfx950.
//
// Per request: the state s = -(e_{t-1} + e_{t-2}) / 2 of the last two
// verification rounds' entropies and z = (B_{t-1}, F_{t-1}) (previous block
// size, full acceptance); then the candidate block size B maximising
// V_B(s, z) - rho_C T_C(B), the V table looked up by (B, s bin, index of
// B_{t-1} among the candidates, F).  Then the requests are grouped by their
// planned size: a stable counting sort.
//
// One work group of 1024 threads does the whole batch in one launch, so a
// serving loop can keep the decision on the device (no host round trip
// between verification and the next round's batching).  Pass 1 decides each
// request (one thread per request, strided) and counts the buckets in LDS;
// pass 2 walks the requests again in tiles of 1024, in order, and places each
// at its bucket's running offset plus its rank among the tile's earlier
// requests of the same bucket (wave ballots, then per-wave counts), which
// keeps the order stable.
//
// Every value that decides an integer is computed in fp32 with one rounding
// per operation (no contraction into fused multiply-adds), ties going to the
// smaller block.
#include "rg_internal.h"

namespace rg {
namespace {

constexpr int kThreads = 1024;
constexpr int kWavesBS = kThreads / 64;

__device__ int decide(const BlockSizeArgs& a, int r) {
#pragma clang fp contract(off)
  const float e1 = a.accept_entropy[r], e2 = a.entropy_hist[r];
  const int prev = a.prev_block[r];
  const float s = -((e1 + e2) * 0.5f);
  int zb = 0;
  for (int i = 0; i < a.nb; ++i)
    if (a.cand[i] <= prev) zb = i;
  const int full = a.accept_len[r] >= prev ? 1 : 0;
  int k = 0;
  for (int i = 0; i + 1 < a.ns; ++i) k += a.edges[i] <= s ? 1 : 0;
  const float* v = a.value + ((size_t)k * a.nb + zb) * 2 + full;  // + b * ns * nb * 2
  const size_t bstride = (size_t)a.ns * a.nb * 2;
  int best = 0;
  float best_u = v[0] - a.rho * a.cost[0];
  for (int b = 1; b < a.nb; ++b) {
    const float u = v[b * bstride] - a.rho * a.cost[b];
    if (u > best_u) {
      best = b;
      best_u = u;
    }
  }
  return best;
}

__global__ __launch_bounds__(kThreads) void plan_block_sizes_kernel(BlockSizeArgs a) {
  __shared__ uint8_t bucket[kMaxBucketRequests];
  __shared__ int count[kMaxBlockCandidates];
  __shared__ int run[kMaxBlockCandidates];
  __shared__ int wave_count[kWavesBS][kMaxBlockCandidates];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < kMaxBlockCandidates) count[tid] = 0;
  __syncthreads();
  for (int r = tid; r < a.num_req; r += kThreads) {
    const int b = decide(a, r);
    a.next_block[r] = a.cand[b];
    a.entropy_hist[r] = a.accept_entropy[r];
    bucket[r] = (uint8_t)b;
    atomicAdd(&count[b], 1);
  }
  if (a.bucket_offsets == nullptr) return;  // uniform: no grouping asked for
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int b = 0; b < a.nb; ++b) {
      run[b] = acc;
      a.bucket_offsets[b] = acc;
      acc += count[b];
    }
    a.bucket_offsets[a.nb] = acc;
  }
  __syncthreads();
  for (int t0 = 0; t0 < a.num_req; t0 += kThreads) {
    const int r = t0 + tid;
    const int b = r < a.num_req ? (int)bucket[r] : -1;
    int rank = 0;
    for (int c = 0; c < a.nb; ++c) {
      const unsigned long long m = __ballot(b == c);
      if (b == c) rank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (lane == 0) wave_count[wave][c] = (int)__popcll(m);
    }
    __syncthreads();
    if (b >= 0) {
      int pos = run[b] + rank;
      for (int w = 0; w < wave; ++w) pos += wave_count[w][b];
      a.order[pos] = r;
    }
    __syncthreads();
    if (tid < a.nb) {
      int add = 0;
      for (int w = 0; w < kWavesBS; ++w) add += wave_count[w][tid];
      run[tid] += add;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_plan_block_sizes(const BlockSizeArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(plan_block_sizes_kernel, dim3(1), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rg

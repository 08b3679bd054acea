// Branch planning and reuse matching of the predictive draft-verify overlap
// (Sec. 5.1), gfx950.
//
// Planning: each request's draft block marks the positions whose draft
// margin P_1st - P_2nd is below delta as risky; the earliest two give
// correction branches (the draft token there replaced by its second
// candidate), and a continuation branch (the whole block accepted) is
// prepared when at most two positions are risky.  One wave per request: each
// pass tests 64 positions with one ballot, whose set bits give the count and
// the earliest positions directly.
//
// Matching: a correction branch is reused when the verifier accepted exactly
// up to its position and produced its replacement token there; the
// continuation when the whole block was accepted and the verifier's bonus
// token is the branch's first token.  One thread per request.
#include "rg_internal.h"

namespace rg {
namespace {

constexpr int kPlanWaves = 4;

__global__ __launch_bounds__(64 * kPlanWaves) void plan_branches_kernel(PlanBranchArgs a) {
  const int r = (int)blockIdx.x * kPlanWaves + (int)(threadIdx.x >> 6);  // wave-uniform
  if (r >= a.num_req) return;
  const int lane = threadIdx.x & 63;
  const int k0 = a.row_indptr[r], n = a.row_indptr[r + 1] - k0;
  int count = 0, p0 = -1, p1 = -1;
  for (int i0 = 0; i0 < n; i0 += 64) {
    const int i = i0 + lane;
    const bool risky = i < n && a.margin[k0 + i] < a.delta;
    unsigned long long bal = __ballot(risky);
    count += __popcll(bal);
    if (p0 < 0 && bal) {
      p0 = i0 + __ffsll((long long)bal) - 1;
      bal &= bal - 1;
    }
    if (p1 < 0 && bal) p1 = i0 + __ffsll((long long)bal) - 1;
  }
  if (lane == 0) {
    a.n_risky[r] = count;
    a.n_corr[r] = min(count, 2);
    a.corr_pos[2 * r] = p0;
    a.corr_pos[2 * r + 1] = p1;
    a.corr_tok[2 * r] = p0 >= 0 ? a.top2[k0 + p0] : -1;
    a.corr_tok[2 * r + 1] = p1 >= 0 ? a.top2[k0 + p1] : -1;
    a.continuation[r] = count <= 2 ? 1 : 0;
  }
}

__global__ __launch_bounds__(256) void match_branches_kernel(MatchBranchArgs a) {
  const int r = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (r >= a.num_req) return;
  const int acc = a.accept_len[r], nt = a.next_token[r], nc = a.n_corr[r];
  int res = -1;
  for (int c = 0; c < 2; ++c)
    if (c < nc && acc == a.corr_pos[2 * r + c] && nt == a.corr_tok[2 * r + c]) res = c;
  if (a.continuation[r] != 0 && acc == a.block_len[r] && nt == a.cont_first[r]) res = nc;
  a.reused[r] = res;
}

}  // namespace

hipError_t launch_plan_branches(const PlanBranchArgs& a, hipStream_t stream) {
  const int blocks = (a.num_req + kPlanWaves - 1) / kPlanWaves;
  hipLaunchKernelGGL(plan_branches_kernel, dim3(blocks), dim3(64 * kPlanWaves), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_match_branches(const MatchBranchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(match_branches_kernel, dim3((a.num_req + 255) / 256), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rg

// Vocabulary-row reductions of one draft-verify round (gfx950).
//
// Verify rows (Sec. 3.1, greedy verification): per row the lowest index of
// the maximum and the entropy of softmax(row); per request the accept length
// (first row whose argmax differs from the token it judges), the verifier's
// token there, and the mean verifier entropy over the rows up to and
// including the first mismatch (e_t of Sec. 5.2).
//
// Draft rows (Sec. 4.1): top-1 / top-2 indices, P_1st, P_2nd, the margin
// P_1st - P_2nd and the entropy.
//
// Both are HBM streams, done in two launches.  The rows kernel gives each
// work group one 8192-entry chunk of one row, held in registers (four
// 16-byte loads per thread), and reduces it to a mergeable state:
//   m = max, i1 = lowest index of m, (v2, i2) = runner-up (draft rows),
//   Z' = sum_{v != i1} exp(x_v - m),  S = sum_v exp(x_v - m) (x_v - m).
// Leaving the top entry's exact 1 out of Z' keeps p1 = 1/(1+Z') and the
// entropy H = log1p(Z') - S/(1+Z') accurate on sharply peaked rows.  Chunk
// states merge exactly: with m = max(m_a, m_b) and the loser's weight
// f = exp(m_lose - m), Z' gains f (1 + Z'_lose) and S gains
// f (S_lose + (m_lose - m)(1 + Z'_lose)); (value, index) pairs merge by value,
// then lower index.  The finalize kernel merges each row's chunk states in a
// fixed order (one wave per row) and, for verify rows, one work group per
// request scans its rows for the first mismatch.  The kernel boundary is the
// only cross-work-group synchronisation: no atomics, no device-scope fences,
// and the workspace needs no initialisation.
#include "rg_internal.h"

namespace rg {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr int kU = kLogitChunk / (8 * kLogitThreads);  // 16-byte loads per thread
constexpr int kE = 8 * kU;                             // entries per thread
constexpr int kNoIndex = 0x7fffffff;
constexpr int kBatchRows = 1024;                       // verify rows scanned per pass

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ __forceinline__ int xcd_item(int grid_items) {
  const int per = grid_items >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

// Vocabulary index of this thread's entry k of the chunk starting at v0.
__device__ __forceinline__ int entry_index(int v0, int k) {
  return v0 + ((k >> 3) * kLogitThreads + (int)threadIdx.x) * 8 + (k & 7);
}

// This thread's entries of chunk [v0, v1) of `row`; entries past v1 are -inf.
__device__ __forceinline__ void load_chunk(const uint16_t* row, int v0, int v1, bool vec, float (&x)[kE]) {
  const int tid = threadIdx.x;
  if (vec && v0 + kLogitChunk <= v1) {
    u32x4 w[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      w[u] = __builtin_nontemporal_load((const u32x4*)(row + v0 + (u * kLogitThreads + tid) * 8));
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[8 * u + 2 * e] = __uint_as_float(w[u][e] << 16);
        x[8 * u + 2 * e + 1] = __uint_as_float(w[u][e] & 0xffff0000u);
      }
    return;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int base = v0 + (u * kLogitThreads + tid) * 8;
    if (vec && base + 8 <= v1) {
      const u32x4 t = *(const u32x4*)(row + base);
      for (int e = 0; e < 4; ++e) {
        x[8 * u + 2 * e] = __uint_as_float(t[e] << 16);
        x[8 * u + 2 * e + 1] = __uint_as_float(t[e] & 0xffff0000u);
      }
    } else {
      for (int j = 0; j < 8; ++j)
        x[8 * u + j] = (base + j < v1) ? __uint_as_float((uint32_t)row[base + j] << 16) : kNegInf;
    }
  }
}

// Work-group reductions over 256 threads (4 waves); every thread gets the
// result.  `red` is an LDS array private to the call site.
__device__ __forceinline__ float wg_max(float v, float* red) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  v = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return v;
}

__device__ __forceinline__ int wg_min(int v, int* red) {
  for (int off = 32; off >= 1; off >>= 1) v = min(v, __shfl_xor(v, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  v = min(min(red[0], red[1]), min(red[2], red[3]));
  __syncthreads();
  return v;
}

// Largest and second largest value of the multiset {a1 >= a2} U {b1 >= b2}.
__device__ __forceinline__ void top2_merge(float& a1, float& a2, float b1, float b2) {
  a2 = fmaxf(fminf(a1, b1), fmaxf(a2, b2));
  a1 = fmaxf(a1, b1);
}

__device__ __forceinline__ void wg_top2(float& v1, float& v2, float* red) {
  for (int off = 32; off >= 1; off >>= 1) {
    const float o1 = __shfl_xor(v1, off), o2 = __shfl_xor(v2, off);
    top2_merge(v1, v2, o1, o2);
  }
  if ((threadIdx.x & 63) == 0) {
    red[2 * (threadIdx.x >> 6)] = v1;
    red[2 * (threadIdx.x >> 6) + 1] = v2;
  }
  __syncthreads();
  v1 = red[0];
  v2 = red[1];
  for (int w = 1; w < 4; ++w) top2_merge(v1, v2, red[2 * w], red[2 * w + 1]);
  __syncthreads();
}

__device__ __forceinline__ void wg_sum2(float& a, float& b, float* red) {
  for (int off = 32; off >= 1; off >>= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  if ((threadIdx.x & 63) == 0) {
    red[2 * (threadIdx.x >> 6)] = a;
    red[2 * (threadIdx.x >> 6) + 1] = b;
  }
  __syncthreads();
  a = (red[0] + red[2]) + (red[4] + red[6]);
  b = (red[1] + red[3]) + (red[5] + red[7]);
  __syncthreads();
}

// Z' (sum of exp(x - m) over entries other than index `top`) and
// sum exp(x - m) * t with t = (x - m) log2(e).  Only the wave holding `top`
// pays for excluding it.
template <bool TAIL>
__device__ __forceinline__ void exp_sums(const float (&x)[kE], int v0, float m, int top, float& z, float& s) {
  const float mc = m * kLog2e;
  int kt = -1;  // position of `top` among this thread's entries
  {
    const int rel = top - v0 - (int)threadIdx.x * 8;
    if (rel >= 0 && (rel % (kLogitThreads * 8)) < 8 && rel / (kLogitThreads * 8) < kU)
      kt = 8 * (rel / (kLogitThreads * 8)) + rel % (kLogitThreads * 8);
  }
  z = 0.f;
  s = 0.f;
  if (__any(kt >= 0)) {
#pragma unroll
    for (int k = 0; k < kE; ++k) {
      float t = __builtin_fmaf(x[k], kLog2e, -mc);
      if (TAIL) t = fmaxf(t, -1000.f);  // entries past the row end are -inf
      const float e = (k == kt) ? 0.f : __builtin_amdgcn_exp2f(t);
      z += e;
      s = __builtin_fmaf(e, t, s);
    }
  } else {
#pragma unroll
    for (int k = 0; k < kE; ++k) {
      float t = __builtin_fmaf(x[k], kLog2e, -mc);
      if (TAIL) t = fmaxf(t, -1000.f);
      const float e = __builtin_amdgcn_exp2f(t);
      z += e;
      s = __builtin_fmaf(e, t, s);
    }
  }
}

struct ChunkRed {
  float f[8];
  int i[4];
};

// One chunk of one row -> (m, i1, v2, i2, Z', S).
template <bool DRAFT>
__device__ __forceinline__ void chunk_state(const uint16_t* row, int v0, int v1, bool vec, ChunkRed& red,
                                            float& m, int& i1, float& v2, int& i2, float& z, float& s) {
  float x[kE];
  load_chunk(row, v0, v1, vec, x);

  float a1 = kNegInf, a2 = kNegInf;
#pragma unroll
  for (int k = 0; k < kE; ++k) {
    if (DRAFT) a2 = fmaxf(a2, fminf(a1, x[k]));
    a1 = fmaxf(a1, x[k]);
  }
  if (DRAFT) wg_top2(a1, a2, red.f);  // a1 = chunk max, a2 = runner-up value (== a1 on a tie)
  else a1 = wg_max(a1, red.f);
  m = a1;
  int idx = kNoIndex;  // lowest index holding m
  for (int k = 0; k < kE; ++k)
    if (x[k] == m) { idx = entry_index(v0, k); break; }
  i1 = wg_min(idx, red.i);
  v2 = kNegInf;
  i2 = kNoIndex;
  if (DRAFT) {
    v2 = a2;
    int j = kNoIndex;
    for (int k = 0; k < kE; ++k)
      if (x[k] == v2 && entry_index(v0, k) != i1) { j = entry_index(v0, k); break; }
    i2 = wg_min(j, red.i);
  }
  if (v0 + kLogitChunk > v1) exp_sums<true>(x, v0, m, i1, z, s);
  else exp_sums<false>(x, v0, m, i1, z, s);
  wg_sum2(z, s, red.f);
  s *= kLn2;
}

struct State {
  float m;
  int i1;
  float v2;
  int i2;
  float zp;
  float s;
};

__device__ __forceinline__ State merge(const State& a, const State& b) {
  const bool a_wins = better(a.m, a.i1, b.m, b.i1);
  const State& w = a_wins ? a : b;
  const State& l = a_wins ? b : a;
  State o = w;
  if (better(l.m, l.i1, w.v2, w.i2)) { o.v2 = l.m; o.i2 = l.i1; }
  if (l.m != kNegInf) {
    const float d = l.m - w.m;
    const float f = __builtin_amdgcn_exp2f(d * kLog2e);
    const float zl = 1.f + l.zp;
    o.zp = w.zp + f * zl;
    o.s = w.s + f * (l.s + d * zl);
  }
  return o;
}

__device__ __forceinline__ State shfl_state(const State& x, int off) {
  return State{__shfl_xor(x.m, off), __shfl_xor(x.i1, off), __shfl_xor(x.v2, off),
               __shfl_xor(x.i2, off), __shfl_xor(x.zp, off), __shfl_xor(x.s, off)};
}

// One wave merges `count` states: lane k takes states k, k+64, ... in order,
// then a fixed butterfly combines the lanes.  Every lane ends with the result.
template <typename Fetch>
__device__ __forceinline__ State wave_merge(int count, Fetch fetch) {
  const int lane = threadIdx.x & 63;
  State acc{kNegInf, kNoIndex, kNegInf, kNoIndex, 0.f, 0.f};
  for (int k = lane; k < count; k += 64) acc = merge(acc, fetch(k));
  for (int off = 1; off < 64; off <<= 1) {
    const State o = shfl_state(acc, off);
    acc = (lane & off) ? merge(o, acc) : merge(acc, o);  // same operand order in both partners
  }
  return acc;
}

__device__ __forceinline__ float entropy_of(const State& st) { return log1pf(st.zp) - st.s / (1.f + st.zp); }

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kLogitThreads) void verify_rows_kernel(VerifyArgs a) {
  __shared__ ChunkRed red;
  const int item = xcd_item(a.grid_rows);
  if (item >= a.rows * a.nchunk) return;
  const int row = item / a.nchunk, c = item % a.nchunk;
  const int v0 = c * kLogitChunk, v1 = min(a.vocab, v0 + kLogitChunk);
  float m, v2, z, s;
  int i1, i2;
  chunk_state<false>(a.logits + (size_t)row * a.row_stride, v0, v1, a.vec != 0, red, m, i1, v2, i2, z, s);
  if (threadIdx.x == 0) a.chunk_st[(size_t)row * a.nchunk + c] = make_float4(m, __int_as_float(i1), z, s);
}

__global__ __launch_bounds__(kLogitThreads) void verify_finalize_kernel(VerifyArgs a) {
  __shared__ int s_am[kBatchRows];
  __shared__ float s_h[kBatchRows];
  const int r = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int k0 = a.row_indptr[r], k1 = a.row_indptr[r + 1];
  const int nrows = k1 - k0;
  int acc_len = nrows;  // kept by wave 0
  int next = -1;
  bool found = false;
  float hsum = 0.f;
  for (int b0 = 0; b0 < nrows; b0 += kBatchRows) {
    const int nb = min(kBatchRows, nrows - b0);
    for (int i = wave; i < nb; i += kLogitThreads / 64) {
      const int row = k0 + b0 + i;
      const float4* cs = a.chunk_st + (size_t)row * a.nchunk;
      const State st = wave_merge(a.nchunk, [&](int k) {
        const float4 q = cs[k];
        return State{q.x, __float_as_int(q.y), kNegInf, kNoIndex, q.z, q.w};
      });
      if (lane == 0) {
        const float h = entropy_of(st);
        a.row_argmax[row] = st.i1;
        if (a.row_entropy) a.row_entropy[row] = h;
        s_am[i] = st.i1;
        s_h[i] = h;
      }
    }
    __syncthreads();
    if (wave == 0 && !found) {
      // first mismatch within this batch, and the entropy sum up to and including it
      for (int j0 = 0; j0 < nb && !found; j0 += 64) {
        const int j = j0 + lane;
        bool mis = false;
        float h = 0.f;
        if (j < nb) {
          const int tok = a.tokens[k0 + b0 + j];
          mis = tok < 0 || s_am[j] != tok;
          h = s_h[j];
        }
        const unsigned long long bal = __ballot(mis);
        const int first = bal ? __ffsll((long long)bal) - 1 : 64;
        float hs = (j < nb && lane <= first) ? h : 0.f;
        for (int off = 32; off >= 1; off >>= 1) hs += __shfl_xor(hs, off);
        hsum += hs;
        if (bal) {
          found = true;
          acc_len = b0 + j0 + first;
          next = s_am[j0 + first];
        }
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    a.accept_len[r] = acc_len;
    a.next_token[r] = next;
    if (a.accept_entropy) a.accept_entropy[r] = nrows ? hsum / (float)(min(acc_len, nrows - 1) + 1) : 0.f;
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kLogitThreads) void draft_rows_kernel(DraftArgs a) {
  __shared__ ChunkRed red;
  const int item = xcd_item(a.grid_rows);
  if (item >= a.rows * a.nchunk) return;
  const int row = item / a.nchunk, c = item % a.nchunk;
  const int v0 = c * kLogitChunk, v1 = min(a.vocab, v0 + kLogitChunk);
  float m, v2, z, s;
  int i1, i2;
  chunk_state<true>(a.logits + (size_t)row * a.row_stride, v0, v1, a.vec != 0, red, m, i1, v2, i2, z, s);
  if (threadIdx.x == 0) {
    const size_t at = (size_t)row * a.nchunk + c;
    a.chunk_a[at] = make_float4(m, __int_as_float(i1), v2, __int_as_float(i2));
    a.chunk_b[at] = make_float2(z, s);
  }
}

__global__ __launch_bounds__(kLogitThreads) void draft_finalize_kernel(DraftArgs a) {
  const int row = blockIdx.x * (kLogitThreads / 64) + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const float4* ca = a.chunk_a + (size_t)row * a.nchunk;
  const float2* cb = a.chunk_b + (size_t)row * a.nchunk;
  const State st = wave_merge(a.nchunk, [&](int k) {
    const float4 q = ca[k];
    const float2 w = cb[k];
    return State{q.x, __float_as_int(q.y), q.z, __float_as_int(q.w), w.x, w.y};
  });
  if ((threadIdx.x & 63) == 0) {
    const float zinv = 1.f / (1.f + st.zp);
    const float d2 = st.v2 - st.m;  // <= 0
    a.top1[row] = st.i1;
    a.top2[row] = st.i2;
    a.p1[row] = zinv;
    a.p2[row] = __expf(d2) * zinv;
    if (a.margin) a.margin[row] = -expm1f(d2) * zinv;
    if (a.entropy) a.entropy[row] = entropy_of(st);
  }
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream) {
  if (a.grid_rows > 0) {
    hipLaunchKernelGGL(verify_rows_kernel, dim3(a.grid_rows), dim3(kLogitThreads), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(verify_finalize_kernel, dim3(a.num_req), dim3(kLogitThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_draft(const DraftArgs& a, hipStream_t stream) {
  if (a.grid_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(draft_rows_kernel, dim3(a.grid_rows), dim3(kLogitThreads), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(draft_finalize_kernel, dim3((a.rows + 3) / 4), dim3(kLogitThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rg

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
// Both passes are HBM streams.  A work group reduces one 8192-entry chunk of
// one row held in registers (four 16-byte loads per thread): first the
// maximum and its lowest index (and the runner-up for draft rows), then
//   Z' = sum_{v != top} exp(x_v - m),  S = sum_v exp(x_v - m) (x_v - m),
// with exp evaluated as exp2 of a log2(e)-scaled difference.  Keeping the top
// element's exact 1 out of Z' keeps p1 = 1/(1+Z') and the entropy
// H = log1p(Z') - S/(1+Z') accurate on sharply peaked rows.  Chunk states
// merge exactly: with m = max(m_a, m_b) and the loser's weight
// f = exp(m_lose - m), Z' gains f (1 + Z'_lose) and S gains
// f (S_lose + (m_lose - m)(1 + Z'_lose)); the (value, index) pairs merge by
// value, then lower index.  The last work group to finish a row (an atomic
// counter in the workspace) merges its chunk states in a fixed order and
// writes the row outputs; for verify rows the last row of a request to
// finish then computes the request's acceptance.  Counters are reset to zero
// by the work group that consumed them.
#include "rg_internal.h"

namespace rg {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr int kU = kLogitChunk / (8 * kLogitThreads);  // 16-byte loads per thread
constexpr int kE = 8 * kU;                             // entries per thread
constexpr int kNoIndex = 0x7fffffff;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ int xcd_item(int grid_items) {
  const int per = grid_items >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

// Loads this thread's entries of chunk [v0, v1) of `row`; entries past v1
// become -inf.  Entry (u, j) has vocabulary index v0 + (u*256 + tid)*8 + j.
__device__ __forceinline__ void load_chunk(const uint16_t* row, int v0, int v1, bool vec, float (&x)[kE]) {
  const int tid = threadIdx.x;
  u32x4 w[kU];
  const bool full = v0 + kLogitChunk <= v1;
  if (vec && full) {
#pragma unroll
    for (int u = 0; u < kU; ++u) w[u] = __builtin_nontemporal_load((const u32x4*)(row + v0 + (u * kLogitThreads + tid) * 8));
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[8 * u + 2 * e] = bf16_to_f32(w[u][e] & 0xffffu);
        x[8 * u + 2 * e + 1] = __uint_as_float(w[u][e] & 0xffff0000u);
      }
  } else {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int base = v0 + (u * kLogitThreads + tid) * 8;
      if (vec && base + 8 <= v1) {
        u32x4 t = *(const u32x4*)(row + base);
        for (int e = 0; e < 4; ++e) {
          x[8 * u + 2 * e] = bf16_to_f32(t[e] & 0xffffu);
          x[8 * u + 2 * e + 1] = __uint_as_float(t[e] & 0xffff0000u);
        }
      } else {
        for (int j = 0; j < 8; ++j) x[8 * u + j] = (base + j < v1) ? bf16_to_f32(row[base + j]) : kNegInf;
      }
    }
  }
}

__device__ __forceinline__ int entry_index(int v0, int k) {
  return v0 + ((k >> 3) * kLogitThreads + (int)threadIdx.x) * 8 + (k & 7);
}

// Sum of exp(x - m) over entries other than index `top`, and of
// exp(x - m) * (x - m) (returned in log2 units: sum e * t with t = (x-m) log2 e).
__device__ __forceinline__ void exp_sums(const float (&x)[kE], int v0, float m, int top, bool tail,
                                         float& z, float& s) {
  const float mc = m * kLog2e;
  // position of `top` among this thread's entries, or -1
  int kt = -1;
  {
    const int rel = top - v0 - (int)threadIdx.x * 8;
    if (rel >= 0 && (rel % (kLogitThreads * 8)) < 8) {
      const int u = rel / (kLogitThreads * 8);
      if (u < kU) kt = 8 * u + (rel % (kLogitThreads * 8));
    }
  }
  z = 0.f;
  s = 0.f;
#pragma unroll
  for (int k = 0; k < kE; ++k) {
    float t = __builtin_fmaf(x[k], kLog2e, -mc);
    if (tail) t = fmaxf(t, -1000.f);  // entries past the row end are -inf
    float e = __builtin_amdgcn_exp2f(t);
    e = (k == kt) ? 0.f : e;
    z += e;
    s = __builtin_fmaf(e, t, s);
  }
}

// Work-group reductions (256 threads).  `red` must hold 4 slots per value.
__device__ __forceinline__ void wg_best(float& v, int& i, float* redf, int* redi) {
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(i, off);
    if (better(ov, oi, v, i)) { v = ov; i = oi; }
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { redf[wave] = v; redi[wave] = i; }
  __syncthreads();
  v = redf[0];
  i = redi[0];
  for (int w = 1; w < 4; ++w)
    if (better(redf[w], redi[w], v, i)) { v = redf[w]; i = redi[w]; }
  __syncthreads();
}

__device__ __forceinline__ void wg_sum2(float& a, float& b, float* red) {
  for (int off = 32; off >= 1; off >>= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { red[2 * wave] = a; red[2 * wave + 1] = b; }
  __syncthreads();
  a = (red[0] + red[2]) + (red[4] + red[6]);
  b = (red[1] + red[3]) + (red[5] + red[7]);
  __syncthreads();
}

// Merge of chunk states (exact up to fp32 rounding).  S is in natural units.
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
  State o;
  o.m = __shfl_xor(x.m, off);
  o.i1 = __shfl_xor(x.i1, off);
  o.v2 = __shfl_xor(x.v2, off);
  o.i2 = __shfl_xor(x.i2, off);
  o.zp = __shfl_xor(x.zp, off);
  o.s = __shfl_xor(x.s, off);
  return o;
}

// Wave 0 merges `count` states; lane k takes states k, k+64, ... in order,
// then a fixed butterfly combines the lanes.  Every lane ends with the result.
template <typename Fetch>
__device__ __forceinline__ State wave_merge(int count, Fetch fetch) {
  const int lane = threadIdx.x & 63;
  State acc{kNegInf, kNoIndex, kNegInf, kNoIndex, 0.f, 0.f};
  for (int k = lane; k < count; k += 64) acc = merge(acc, fetch(k));
  for (int off = 1; off < 64; off <<= 1) {
    const State o = shfl_state(acc, off);
    // order the operands by lane so both partners compute the same value
    acc = (lane & off) ? merge(o, acc) : merge(acc, o);
  }
  return acc;
}

__device__ __forceinline__ float row_entropy_of(const State& st) {
  const float z = 1.f + st.zp;
  return log1pf(st.zp) - st.s / z;
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kLogitThreads) void verify_kernel(VerifyArgs a) {
  __shared__ float redf[8];
  __shared__ int redi[4];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= a.grid_rows) {
    // requests without verify rows
    const int r = ((int)blockIdx.x - a.grid_rows) * kLogitThreads + tid;
    if (r < a.num_req && a.row_indptr[r + 1] == a.row_indptr[r]) {
      a.accept_len[r] = 0;
      a.next_token[r] = -1;
      if (a.accept_entropy) a.accept_entropy[r] = 0.f;
    }
    return;
  }
  const int item = xcd_item(a.grid_rows);
  if (item >= a.rows * a.nchunk) return;
  const int row = item / a.nchunk, c = item % a.nchunk;
  const int v0 = c * kLogitChunk, v1 = min(a.vocab, v0 + kLogitChunk);
  const bool tail = v0 + kLogitChunk > v1;

  float x[kE];
  load_chunk(a.logits + (size_t)row * a.row_stride, v0, v1, a.vec != 0, x);

  // request owning this row: number of row_indptr[1..R] entries <= row
  int req = 0, k0 = 0, k1 = 0;
  if (tid < 64) {
    int cnt = 0;
    for (int j0 = 1; j0 <= a.num_req; j0 += 64) {
      const int j = j0 + tid;
      const int v = (j <= a.num_req) ? a.row_indptr[j] : 0x7fffffff;
      cnt += __popcll(__ballot(v <= row));
    }
    req = min(cnt, a.num_req - 1);
    k0 = a.row_indptr[req];
    k1 = a.row_indptr[req + 1];
  }

  float bv = kNegInf;
  int bi = kNoIndex;
#pragma unroll
  for (int k = 0; k < kE; ++k)
    if (x[k] > bv) { bv = x[k]; bi = entry_index(v0, k); }
  wg_best(bv, bi, redf, redi);

  float z, s;
  exp_sums(x, v0, bv, bi, tail, z, s);
  wg_sum2(z, s, redf);

  if (tid == 0) {
    a.chunk_st[(size_t)row * a.nchunk + c] = make_float4(bv, __int_as_float(bi), z, s * kLn2);
    __threadfence();
    s_flag = (atomicAdd(&a.row_cnt[row], 1) == a.nchunk - 1);
  }
  __syncthreads();
  if (!s_flag || tid >= 64) return;

  // last chunk of this row: merge its chunk states
  __threadfence();
  const float4* cs = a.chunk_st + (size_t)row * a.nchunk;
  const State st = wave_merge(a.nchunk, [&](int k) {
    const float4 q = cs[k];
    return State{q.x, __float_as_int(q.y), kNegInf, kNoIndex, q.z, q.w};
  });
  const float h = row_entropy_of(st);
  int last_row = 0;
  if (tid == 0) {
    a.row_argmax[row] = st.i1;
    if (a.row_entropy) a.row_entropy[row] = h;
    a.row_st[row] = make_float2(__int_as_float(st.i1), h);
    a.row_cnt[row] = 0;
    __threadfence();
    last_row = (atomicAdd(&a.req_cnt[req], 1) == (k1 - k0) - 1);
  }
  // wave 0 only from here on (tid < 64)
  if (!__shfl(last_row, 0)) return;

  // last row of request `req`: greedy acceptance
  __threadfence();
  const int nrows = k1 - k0;
  int acc_len = nrows;
  for (int b = 0; b < nrows; b += 64) {
    const int k = b + tid;
    bool mismatch = false;
    if (k < nrows) {
      const int tok = a.tokens[k0 + k];
      const int am = __float_as_int(a.row_st[k0 + k].x);
      mismatch = tok < 0 || am != tok;
    }
    const unsigned long long bal = __ballot(mismatch);
    if (bal) { acc_len = b + __ffsll((long long)bal) - 1; break; }
  }
  const int last = min(acc_len, nrows - 1);
  float hs = 0.f;
  for (int k = tid; k <= last; k += 64) hs += a.row_st[k0 + k].y;
  for (int off = 32; off >= 1; off >>= 1) hs += __shfl_xor(hs, off);
  if (tid == 0) {
    a.accept_len[req] = acc_len;
    a.next_token[req] = acc_len < nrows ? __float_as_int(a.row_st[k0 + acc_len].x) : -1;
    if (a.accept_entropy) a.accept_entropy[req] = hs / (float)(last + 1);
    a.req_cnt[req] = 0;
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kLogitThreads) void draft_kernel(DraftArgs a) {
  __shared__ float redf[8];
  __shared__ int redi[4];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  const int item = xcd_item(a.grid_rows);
  if (item >= a.rows * a.nchunk) return;
  const int row = item / a.nchunk, c = item % a.nchunk;
  const int v0 = c * kLogitChunk, v1 = min(a.vocab, v0 + kLogitChunk);
  const bool tail = v0 + kLogitChunk > v1;

  float x[kE];
  load_chunk(a.logits + (size_t)row * a.row_stride, v0, v1, a.vec != 0, x);

  // per-thread top two (value desc, index asc); entries scanned in index order
  float b1 = kNegInf, b2 = kNegInf;
  int i1 = kNoIndex, i2 = kNoIndex;
#pragma unroll
  for (int k = 0; k < kE; ++k) {
    const float v = x[k];
    const int idx = entry_index(v0, k);
    if (v > b1) { b2 = b1; i2 = i1; b1 = v; i1 = idx; }
    else if (v > b2) { b2 = v; i2 = idx; }
  }
  // work-group merge of the top-two lists
  {
    for (int off = 32; off >= 1; off >>= 1) {
      const float o1 = __shfl_xor(b1, off), o2 = __shfl_xor(b2, off);
      const int oi1 = __shfl_xor(i1, off), oi2 = __shfl_xor(i2, off);
      if (better(b1, i1, o1, oi1)) {
        if (better(o1, oi1, b2, i2)) { b2 = o1; i2 = oi1; }
      } else {
        if (better(b1, i1, o2, oi2)) { b2 = b1; i2 = i1; } else { b2 = o2; i2 = oi2; }
        b1 = o1; i1 = oi1;
      }
    }
    __shared__ float t1v[4], t2v[4];
    __shared__ int t1i[4], t2i[4];
    const int wave = tid >> 6;
    if ((tid & 63) == 0) { t1v[wave] = b1; t1i[wave] = i1; t2v[wave] = b2; t2i[wave] = i2; }
    __syncthreads();
    b1 = t1v[0]; i1 = t1i[0]; b2 = t2v[0]; i2 = t2i[0];
    for (int w = 1; w < 4; ++w) {
      const float o1 = t1v[w], o2 = t2v[w];
      const int oi1 = t1i[w], oi2 = t2i[w];
      if (better(b1, i1, o1, oi1)) {
        if (better(o1, oi1, b2, i2)) { b2 = o1; i2 = oi1; }
      } else {
        if (better(b1, i1, o2, oi2)) { b2 = b1; i2 = i1; } else { b2 = o2; i2 = oi2; }
        b1 = o1; i1 = oi1;
      }
    }
    __syncthreads();
  }

  float z, s;
  exp_sums(x, v0, b1, i1, tail, z, s);
  wg_sum2(z, s, redf);

  if (tid == 0) {
    const size_t at = (size_t)row * a.nchunk + c;
    a.chunk_a[at] = make_float4(b1, __int_as_float(i1), b2, __int_as_float(i2));
    a.chunk_b[at] = make_float2(z, s * kLn2);
    __threadfence();
    s_flag = (atomicAdd(&a.row_cnt[row], 1) == a.nchunk - 1);
  }
  __syncthreads();
  if (!s_flag || tid >= 64) return;

  __threadfence();
  const float4* ca = a.chunk_a + (size_t)row * a.nchunk;
  const float2* cb = a.chunk_b + (size_t)row * a.nchunk;
  const State st = wave_merge(a.nchunk, [&](int k) {
    const float4 q = ca[k];
    const float2 w = cb[k];
    return State{q.x, __float_as_int(q.y), q.z, __float_as_int(q.w), w.x, w.y};
  });
  if (tid == 0) {
    const float zinv = 1.f / (1.f + st.zp);
    const float d2 = st.v2 - st.m;  // <= 0
    a.top1[row] = st.i1;
    a.top2[row] = st.i2;
    a.p1[row] = zinv;
    a.p2[row] = __expf(d2) * zinv;
    if (a.margin) a.margin[row] = -expm1f(d2) * zinv;
    if (a.entropy) a.entropy[row] = row_entropy_of(st);
    a.row_cnt[row] = 0;
  }
}

__global__ void zero_kernel(uint4* p, size_t n16, uint8_t* tail, size_t ntail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream) {
  const int extra = (a.num_req + kLogitThreads - 1) / kLogitThreads;
  hipLaunchKernelGGL(verify_kernel, dim3(a.grid_rows + extra), dim3(kLogitThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_draft(const DraftArgs& a, hipStream_t stream) {
  if (a.grid_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(draft_kernel, dim3(a.grid_rows), dim3(kLogitThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16, ntail = bytes % 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks == 0) blocks = 1;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, (uint4*)ptr, n16,
                     (uint8_t*)ptr + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace rg

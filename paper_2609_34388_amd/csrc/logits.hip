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
// fixed order (a group of lanes per row, all states fetched at once) and, for
// verify rows, one work group per request scans its rows for the first
// mismatch.  The kernel boundary is the
// only cross-work-group synchronisation: no atomics, no device-scope fences,
// and the workspace needs no initialisation.
#include <mutex>

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
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ __forceinline__ int xcd_item(int grid_items) {
  const int per = grid_items >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

// Maximum and median of loaded values through the instructions themselves:
// fmaxf / fmed3 on values the compiler cannot prove canonical get a quieting
// v_max_f32 x, x, x per input first (one more instruction per entry).  The
// inputs here are finite or -inf (padding), where the two agree.
__device__ __forceinline__ float max3_of(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max2_of(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float med3_of(float a, float b, float c) {
  float r;
  asm("v_med3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Vocabulary index of this thread's entry k of the chunk starting at v0.
__device__ __forceinline__ int entry_index(int v0, int k) {
  return v0 + ((k >> 3) * kLogitThreads + (int)threadIdx.x) * 8 + (k & 7);
}

// bf16 -> fp32 of 8 packed values (two shifts per pair).
__device__ __forceinline__ void widen8(u32x4 w, float* x) {
  const f32x8 f = __builtin_convertvector(__builtin_bit_cast(bf16x8, w), f32x8);
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = f[j];
}

// This thread's entries of chunk [v0, v1) of `row`; entries past v1 are -inf.
__device__ __forceinline__ void load_chunk(const uint16_t* row, int v0, int v1, bool vec, float (&x)[kE]) {
  const int tid = threadIdx.x;
  if (vec && v0 + kLogitChunk <= v1) {
    u32x4 w[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      w[u] = __builtin_nontemporal_load((const u32x4*)(row + v0 + (u * kLogitThreads + tid) * 8));
    // All loads go out before the first use of any: otherwise the scheduler
    // may convert the first load's entries before issuing the others, and the
    // wait for that load costs a second memory round trip.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kU; ++u) widen8(w[u], x + 8 * u);
    return;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int base = v0 + (u * kLogitThreads + tid) * 8;
    if (vec && base + 8 <= v1) {
      widen8(*(const u32x4*)(row + base), x + 8 * u);
    } else {
      for (int j = 0; j < 8; ++j)
        x[8 * u + j] = (base + j < v1) ? (float)__builtin_bit_cast(__bf16, row[base + j]) : kNegInf;
    }
  }
}

template <typename T>
__device__ __forceinline__ T lane_read(T v, int l) {
  if constexpr (sizeof(T) == 4 && __is_same(T, float))
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
  else
    return __builtin_amdgcn_readlane(v, l);
}

// Wave reductions, six instructions with a DPP operand, in place: xor 1,
// xor 2, half-row mirror and row mirror leave every lane of a 16-lane row
// holding its row's result; row_bcast:15 then combines rows 0 and 1 into row
// 1 and rows 2 and 3 into row 3, and row_bcast:31 rows 1 and 3 into row 3,
// so lane 63 holds the wave's result, read once as a scalar.  Each step
// first waits the two wait states a DPP read of a just-written VGPR needs.
// Every lane of the wave must be active.
#define RG_WAVE_REDUCE_ASM(INSN)                                                        \
  "s_nop 1\n " INSN " %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n" \
  "s_nop 1\n " INSN " %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n" \
  "s_nop 1\n " INSN " %0, %0, %0 row_half_mirror row_mask:0xf bank_mask:0xf\n"     \
  "s_nop 1\n " INSN " %0, %0, %0 row_mirror row_mask:0xf bank_mask:0xf\n"          \
  "s_nop 1\n " INSN " %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n"        \
  "s_nop 1\n " INSN " %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf"
__device__ __forceinline__ float wave_sum(float v) {
  asm volatile(RG_WAVE_REDUCE_ASM("v_add_f32_dpp") : "+v"(v));
  return lane_read(v, 63);
}
__device__ __forceinline__ float wave_max(float v) {
  asm volatile(RG_WAVE_REDUCE_ASM("v_max_f32_dpp") : "+v"(v));
  return lane_read(v, 63);
}
__device__ __forceinline__ int wave_isum(int v) {
  asm volatile(RG_WAVE_REDUCE_ASM("v_add_u32_dpp") : "+v"(v));
  return lane_read(v, 63);
}
__device__ __forceinline__ int wave_imin(int v) {
  asm volatile(RG_WAVE_REDUCE_ASM("v_min_i32_dpp") : "+v"(v));
  return lane_read(v, 63);
}
// The two smallest of the lanes' disjoint index pairs {v1 <= v2}: the
// smallest first index, then the smallest of the other lanes' first indices
// and that lane's second one.
__device__ __forceinline__ void wave_min2(int& v1, int& v2) {
  const int a1 = wave_imin(v1);
  v2 = wave_imin(v1 == a1 ? v2 : v1);
  v1 = a1;
}

// Smallest and second smallest of two disjoint sets {a1 <= a2}, {b1 <= b2}.
__device__ __forceinline__ void min2_merge(int& a1, int& a2, int b1, int b2) {
  a2 = min(max(a1, b1), min(a2, b2));
  a1 = min(a1, b1);
}

// Z'' and S partial sums of this thread's entries against the chunk maximum
// m (mc = m log2 e): exp(x - m) and exp(x - m)(x - m) in log2 units, in two
// independent chains to halve the dependent latency.  Entries equal to m
// have been replaced by a stand-in whose terms are exactly 0.  Entries past the
// row end are -inf and only occur in a row's last chunk (TAIL), where t is
// clamped so that e * t stays 0.
template <bool TAIL>
__device__ __forceinline__ void exp_sums(const float (&x)[kE], float mc, float& zz, float& ss) {
  float z0 = 0.f, z1 = 0.f, s0 = 0.f, s1 = 0.f;
#pragma unroll
  for (int k = 0; k < kE; k += 2) {
    float t0 = __builtin_fmaf(x[k], kLog2e, -mc);
    float t1 = __builtin_fmaf(x[k + 1], kLog2e, -mc);
    if (TAIL) {
      t0 = fmaxf(t0, -1000.f);
      t1 = fmaxf(t1, -1000.f);
    }
    const float e0 = __builtin_amdgcn_exp2f(t0);
    const float e1 = __builtin_amdgcn_exp2f(t1);
    z0 += e0;
    z1 += e1;
    s0 = __builtin_fmaf(e0, t0, s0);
    s1 = __builtin_fmaf(e1, t1, s1);
  }
  zz = z0 + z1;
  ss = s0 + s1;
}

struct ChunkRed {
  float m[4];      // per wave: largest value
  float zs[2][4];  // per wave: Z'' and S partial sums
  float c2[4];     // per wave: largest value once one entry holding m is set aside
  int cnt[4];      // per wave: entries equal to the chunk maximum
  int f[2][4];     // per wave: first, second index of the maximum
  int g[4];        // per wave: first index of the runner-up
};

// Sets aside this thread's entries equal to the chunk maximum m: counts
// them, keeps their two lowest indices and replaces them by a stand-in value
// far enough below m that its exponential is exactly 0 and its product with
// the scaled difference stays finite (m - |m|/16 - 256, with the lowest
// mantissa bit set so that it is no bfloat16 value and no input equals it).  Only
// groups where some lane holds m are visited (usually one group of one lane
// per chunk; the test is wave-uniform), in descending order so that the
// lowest index is assigned last.  For draft rows a group's maximum that
// equals m becomes the group's second largest value (m again if m occurs
// twice in it), so that the largest of the thread's group maxima is its
// runner-up whenever the chunk holds m once.
template <bool DRAFT>
__device__ __forceinline__ void set_aside_max(float (&x)[kE], float (&gm)[kU], float m, int v0, int& cnt,
                                              int& f1, int& f2, bool& hit) {
#pragma unroll
  for (int u = kU - 1; u >= 0; --u) {
    if (__any(gm[u] == m)) {
      hit = true;
      const float gone = __int_as_float(__float_as_int(m - (fabsf(m) * 0.0625f + 256.f)) | 1);
      float* y = x + 8 * u;
      float t1 = kNegInf, t2 = kNegInf;  // t1 >= t2: the group's two largest values
#pragma unroll
      for (int j = 7; j >= 0; --j) {
        if (DRAFT) {
          t2 = med3_of(t1, t2, y[j]);
          t1 = max2_of(t1, y[j]);
        }
        const bool eq = y[j] == m;  // selects, not branches: no copies where groups join
        cnt += eq ? 1 : 0;
        f2 = eq ? f1 : f2;
        f1 = eq ? entry_index(v0, 8 * u + j) : f1;
        y[j] = eq ? gone : y[j];
      }
      if (DRAFT && gm[u] == m) gm[u] = t2;
    }
  }
}

// One chunk of one row -> (m, i1, v2, i2, Z', S).  Round 1: the chunk
// maximum m.  Round 2: Z'' = sum of exp(x - m) over entries below m, S, the
// number of entries equal to m and their two lowest indices; for draft rows
// also the runner-up v2 (m again when m occurs twice, else the largest value
// below m).  Round 3 (draft rows with m once): the lowest index holding v2.
// Then Z' (all but the top entry) = Z'' + (count - 1), exactly.  Only thread
// 0 receives (i1, i2, Z', S).
template <bool DRAFT>
__device__ __forceinline__ void chunk_state(const uint16_t* row, int v0, int v1, bool vec, ChunkRed& red,
                                            float& m, int& i1, float& v2, int& i2, float& z, float& s) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float x[kE];
  load_chunk(row, v0, v1, vec, x);

  // Maximum of each group of 8 entries (one 16-byte load: consecutive
  // vocabulary indices) and of this thread's entries.
  float gm[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const float* y = x + 8 * u;
    gm[u] = max3_of(max3_of(y[0], y[1], y[2]), max3_of(y[3], y[4], y[5]), max2_of(y[6], y[7]));
  }
  float a1 = gm[0];
#pragma unroll
  for (int u = 1; u < kU; ++u) a1 = max2_of(a1, gm[u]);
  a1 = wave_max(a1);
  if (lane == 0) red.m[wave] = a1;
  __syncthreads();
  m = max2_of(max2_of(red.m[0], red.m[1]), max2_of(red.m[2], red.m[3]));

  int cnt = 0, f1 = kNoIndex, f2 = kNoIndex;
  bool hit = false;
  set_aside_max<DRAFT>(x, gm, m, v0, cnt, f1, f2, hit);
  float zz, ss, c2 = kNegInf;
  if (v0 + kLogitChunk <= v1) exp_sums<false>(x, m * kLog2e, zz, ss);
  else exp_sums<true>(x, m * kLog2e, zz, ss);
  if (DRAFT) {
    c2 = gm[0];
#pragma unroll
    for (int u = 1; u < kU; ++u) c2 = max2_of(c2, gm[u]);
  }
  zz = wave_sum(zz);
  ss = wave_sum(ss);
  if (DRAFT) c2 = wave_max(c2);
  if (hit) {  // wave-uniform
    cnt = wave_isum(cnt);
    if (DRAFT) wave_min2(f1, f2);
    else f1 = wave_imin(f1);
  }
  if (lane == 0) {
    red.zs[0][wave] = zz;
    red.zs[1][wave] = ss;
    red.c2[wave] = c2;
    red.cnt[wave] = cnt;
    red.f[0][wave] = f1;
    red.f[1][wave] = f2;
  }
  __syncthreads();
  int g = kNoIndex;
  v2 = kNegInf;
  if (DRAFT) {
    cnt = (red.cnt[0] + red.cnt[1]) + (red.cnt[2] + red.cnt[3]);
    v2 = cnt >= 2 ? m : max2_of(max2_of(red.c2[0], red.c2[1]), max2_of(red.c2[2], red.c2[3]));
    if (cnt < 2 && v2 != kNegInf) {  // block-uniform
      // Only groups whose maximum reaches v2 can hold it.
      bool scanned = false;
#pragma unroll
      for (int u = kU - 1; u >= 0; --u) {
        if (__any(gm[u] >= v2)) {
          scanned = true;
#pragma unroll
          for (int j = 7; j >= 0; --j)
            if (x[8 * u + j] == v2) g = entry_index(v0, 8 * u + j);
        }
      }
      if (scanned) g = wave_imin(g);
      if (lane == 0) red.g[wave] = g;
      __syncthreads();
      g = min(min(red.g[0], red.g[1]), min(red.g[2], red.g[3]));
    }
  }
  if (threadIdx.x != 0) return;
  zz = (red.zs[0][0] + red.zs[0][1]) + (red.zs[0][2] + red.zs[0][3]);
  ss = (red.zs[1][0] + red.zs[1][1]) + (red.zs[1][2] + red.zs[1][3]);
  cnt = (red.cnt[0] + red.cnt[1]) + (red.cnt[2] + red.cnt[3]);
  f1 = red.f[0][0];
  f2 = red.f[1][0];
  for (int w = 1; w < kLogitThreads / 64; ++w) {
    if (DRAFT) min2_merge(f1, f2, red.f[0][w], red.f[1][w]);
    else f1 = min(f1, red.f[0][w]);
  }
  i1 = f1;
  i2 = !DRAFT ? kNoIndex : (cnt >= 2 ? f2 : g);
  z = zz + (float)(cnt - 1);
  s = ss * kLn2;
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

// Lanes per row when a row's chunk states are merged by a lane group: the
// smallest power of two >= nchunk, at most 64 (a group never spans waves).
__device__ __forceinline__ int group_lanes(int nchunk) {
  int l = 1;
  while (l < nchunk && l < 64) l <<= 1;
  return l;
}

// A group of `lanes` consecutive lanes merges `count` states: lane j of the
// group takes states j, j + lanes, ... in order, then a fixed butterfly
// combines the group.  Every lane of the group ends with the result.  All
// states of all groups are fetched at once, so a pass costs one round trip.
template <typename Fetch>
__device__ __forceinline__ State group_merge(int lanes, int count, bool active, Fetch fetch) {
  const int j = (threadIdx.x & 63) & (lanes - 1);
  State acc{kNegInf, kNoIndex, kNegInf, kNoIndex, 0.f, 0.f};
  if (active)
    for (int k = j; k < count; k += lanes) acc = merge(acc, fetch(k));
  for (int off = 1; off < lanes; off <<= 1) {
    const State o = shfl_state(acc, off);
    acc = (j & off) ? merge(o, acc) : merge(acc, o);  // same operand order in both partners
  }
  return acc;
}

__device__ __forceinline__ float entropy_of(const State& st) { return log1pf(st.zp) - st.s / (1.f + st.zp); }

// ---------------------------------------------------------------------------
// One (row, chunk) item of the verify rows.
__device__ __forceinline__ void verify_rows(const VerifyArgs& a, int item, ChunkRed& red) {
  const int row = item >> a.cshift, c = item & ((1 << a.cshift) - 1);
  if (c >= a.nchunk) return;  // a slot past the row's last chunk
  const int v0 = c * kLogitChunk, v1 = min(a.vocab, v0 + kLogitChunk);
  float m, v2, z, s;
  int i1, i2;
  chunk_state<false>(a.logits + (size_t)row * a.row_stride, v0, v1, a.vec != 0, red, m, i1, v2, i2, z, s);
  if (threadIdx.x == 0) a.chunk_st[(size_t)row * a.nchunk + c] = make_float4(m, __int_as_float(i1), z, s);
}

__global__ __launch_bounds__(kLogitThreads) void verify_rows_kernel(VerifyArgs a) {
  __shared__ ChunkRed red;
  const int item = xcd_item(a.grid_rows);
  if (item < (a.rows << a.cshift)) verify_rows(a, item, red);
}

struct FinalizeLds {
  int am[kBatchRows];
  float h[kBatchRows];
  int tok[kBatchRows];
};

// Request r of the verify rows: merge each row's chunk states, then the
// first mismatch, next token and e_t.
__device__ __forceinline__ void verify_finalize(const VerifyArgs& a, int r, FinalizeLds& lds) {
  int* s_am = lds.am;
  float* s_h = lds.h;
  int* s_tok = lds.tok;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int k0 = a.row_indptr[r], k1 = a.row_indptr[r + 1];
  const int nrows = k1 - k0;
  const int lanes = group_lanes(a.nchunk);
  const int per_pass = kLogitThreads / lanes;  // rows merged per pass
  int acc_len = nrows;  // kept by wave 0
  int next = -1;
  bool found = false;
  float hsum = 0.f;
  for (int b0 = 0; b0 < nrows; b0 += kBatchRows) {
    const int nb = min(kBatchRows, nrows - b0);
    for (int j = tid; j < nb; j += kLogitThreads) s_tok[j] = a.tokens[k0 + b0 + j];
    for (int i0 = 0; i0 < nb; i0 += per_pass) {
      const int i = i0 + tid / lanes;
      const bool active = i < nb;
      const float4* cs = a.chunk_st + (size_t)(k0 + b0 + (active ? i : 0)) * a.nchunk;
      const State st = group_merge(lanes, a.nchunk, active, [&](int k) {
        const float4 q = cs[k];
        return State{q.x, __float_as_int(q.y), kNegInf, kNoIndex, q.z, q.w};
      });
      if (active && (tid & (lanes - 1)) == 0) {
        const int row = k0 + b0 + i;
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
          const int tok = s_tok[j];
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

__global__ __launch_bounds__(kLogitThreads) void verify_finalize_kernel(VerifyArgs a) {
  __shared__ FinalizeLds lds;
  verify_finalize(a, blockIdx.x, lds);
}

// ---------------------------------------------------------------------------
// One (row, chunk) item of the draft rows.
__device__ __forceinline__ void draft_rows(const DraftArgs& a, int item, ChunkRed& red) {
  const int row = item >> a.cshift, c = item & ((1 << a.cshift) - 1);
  if (c >= a.nchunk) return;  // a slot past the row's last chunk
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

__global__ __launch_bounds__(kLogitThreads) void draft_rows_kernel(DraftArgs a) {
  __shared__ ChunkRed red;
  const int item = xcd_item(a.grid_rows);
  if (item < (a.rows << a.cshift)) draft_rows(a, item, red);
}

// Draft rows blk * (256 / lanes) ...: one lane group per row.
__device__ __forceinline__ void draft_finalize(const DraftArgs& a, int blk) {
  const int lanes = group_lanes(a.nchunk);
  const int row = blk * (kLogitThreads / lanes) + (int)threadIdx.x / lanes;
  const bool active = row < a.rows;
  const size_t base = (size_t)(active ? row : 0) * a.nchunk;
  const State st = group_merge(lanes, a.nchunk, active, [&](int k) {
    const float4 q = a.chunk_a[base + k];
    const float2 w = a.chunk_b[base + k];
    return State{q.x, __float_as_int(q.y), q.z, __float_as_int(q.w), w.x, w.y};
  });
  if (active && (threadIdx.x & (lanes - 1)) == 0) {
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

__global__ __launch_bounds__(kLogitThreads) void draft_finalize_kernel(DraftArgs a) { draft_finalize(a, blockIdx.x); }

// Both passes of one round in two launches: the row items of the verify rows
// and of the draft rows share one grid, and so do the two finalize steps.
__global__ __launch_bounds__(kLogitThreads) void round_rows_kernel(VerifyArgs v, DraftArgs d, int32_t grid) {
  __shared__ ChunkRed red;
  const int item = xcd_item(grid);
  const int nv = v.rows << v.cshift;
  if (item < nv) verify_rows(v, item, red);
  else if (item - nv < (d.rows << d.cshift)) draft_rows(d, item - nv, red);
}

__global__ __launch_bounds__(kLogitThreads) void round_finalize_kernel(VerifyArgs v, DraftArgs d) {
  __shared__ FinalizeLds lds;
  const int b = blockIdx.x;
  if (b < v.num_req) verify_finalize(v, b, lds);
  else draft_finalize(d, b - v.num_req);
}

int draft_finalize_groups(const DraftArgs& a) {
  int lanes = 1;
  while (lanes < a.nchunk && lanes < 64) lanes <<= 1;
  const int rows_per_group = kLogitThreads / lanes;
  return (a.rows + rows_per_group - 1) / rows_per_group;
}

// Scratch of the allocation-free logit round (rg_verify_and_confidence_noalloc):
// the chunk states that rg_verify_and_confidence keeps in its caller's
// workspace.  Every GPU the library runs on holds one copy until the process
// ends; the row passes write every state the finalize pass reads, so nothing
// in it has to start at zero.
__device__ __attribute__((aligned(256))) unsigned char scratch[kNoAllocScratchBytes];

}  // namespace

// Device address of this GPU's copy of `scratch`, looked up once per device
// (with that device current) and kept: in host code the array's name is only
// a host-side stand-in, never a device address.
hipError_t noalloc_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

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
  hipLaunchKernelGGL(draft_finalize_kernel, dim3(draft_finalize_groups(a)), dim3(kLogitThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_round(const VerifyArgs& v, const DraftArgs& d, hipStream_t stream) {
  const int64_t items = ((int64_t)v.rows << v.cshift) + ((int64_t)d.rows << d.cshift);
  const int32_t grid = (int32_t)((items + 7) / 8 * 8);
  if (grid > 0) {
    hipLaunchKernelGGL(round_rows_kernel, dim3(grid), dim3(kLogitThreads), 0, stream, v, d, grid);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int blocks = v.num_req + (d.rows > 0 ? draft_finalize_groups(d) : 0);
  hipLaunchKernelGGL(round_finalize_kernel, dim3(blocks), dim3(kLogitThreads), 0, stream, v, d);
  return hipGetLastError();
}

}  // namespace rg

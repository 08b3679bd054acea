// Hybrid-mask paged attention of one fused draft-verify step (gfx950).
//
// What is computed (Eq. 1, Sec. 3.1, with the prefix = cached context +
// verify rows and the draft set = the next draft block): for request r with
// L cached tokens, V verify rows and B draft rows (n = V + B, T = L + n keys),
// verify row i sees keys j <= L + i and draft rows see all T keys;
// out = softmax(scale * q k^T + mask) v per query head, query head h reading
// KV head h / (Hq / Hkv).
//
// Work decomposition.  A work item is (request, KV head, column group, KV
// chunk).  Its "columns" are all (query token, query head) pairs of the
// request that share the KV head -- n * Hq/Hkv of them -- so every K/V byte
// of a chunk is read from HBM once for all of them.  Each of the 4 waves owns
// one or two 32-column tiles.  Requests whose keys span several chunks write
// un-normalised partial outputs plus (max, sum) per column; a second kernel
// merges them with the usual log-sum-exp weights.
//
// Per 64-key step the work group stages K and V of four 16-token pages into
// LDS (double buffered; the next step's global loads are in flight while the
// current step computes).  On each 32-key sub-tile a wave forms
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K rows are the MFMA rows, query
// columns the MFMA columns), applies the mask, updates the running max and
// sum in fp32 (exp2 with the scale folded in), converts P to bf16 and
// accumulates O^T += V^T P^T with the same MFMA.  The K rows of a sub-tile
// are loaded in a permuted order (bits 2 and 3 of the row index swapped) so
// that the S^T accumulator registers a lane holds are exactly the P^T operand
// the PV MFMA needs and the matching V^T operand is 8 consecutive keys of one
// head dimension: 16 contiguous bytes of a dimension-major V page.
//
// Bounds: a work group loads only keys of its own chunk, which ends at or
// before T, so unused slots of a request's last page are never read; staged
// K rows and V entries past the chunk end are zero-filled and their scores
// masked to -inf.
#include "rg_internal.h"

namespace rg {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ int swap23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Swizzle of the two 16-byte halves of a dimension row of a V page in LDS.
__device__ __forceinline__ int vswz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

__device__ __forceinline__ int find_request(const AttnPlan& p, int item, bool combine) {
  int lo = 0, hi = p.num_req - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    int start = combine ? p.req[mid].comb_start : p.req[mid].item_start;
    if (start <= item) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Consecutive work items of one (request, KV head) land on one XCD: the
// dispatcher deals work groups to the 8 XCDs round-robin, so block b runs on
// XCD b % 8; give XCD x the item range [x*per, (x+1)*per).
__device__ __forceinline__ int xcd_item(int grid_items) {
  const int per = grid_items >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

template <int D, int QTW>
__global__ __launch_bounds__(kAttnThreads) void attn_fwd_kernel(AttnArgs a, AttnPlan p) {
  constexpr int NCH = D / 8;          // 16-byte chunks per K row
  constexpr int KSTEPS = D / 16;      // MFMA k-steps of q.k
  constexpr int DT = D / 32;          // 32-wide head-dim tiles of the output
  constexpr int TILE = kKeyTile * D;  // bf16 elements of one staged K (or V) tile
  constexpr int PER_THREAD = TILE / 8 / kAttnThreads;  // 16-byte chunks per thread
  constexpr int MAXPAGES = kMaxChunkKeys / kPageSize;

  __shared__ __attribute__((aligned(16))) uint16_t lds_k[2][TILE];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v[2][TILE];
  __shared__ int32_t lds_pages[MAXPAGES];

  const int item = xcd_item(p.grid_items);
  if (item >= p.total_items) return;
  const int r = find_request(p, item, false);
  const AttnReq rq = p.req[r];
  const int n = rq.nv & 0xffff, nver = rq.nv >> 16, L = rq.ctx, T = L + n;
  const int g = a.g;
  const int M = n * g;
  const int cols_per_group = 128 * QTW;
  const int ncg = (M + cols_per_group - 1) / cols_per_group;
  const int nch = (T + p.chunk - 1) / p.chunk;
  int local = item - rq.item_start;
  const int c = local % nch;
  local /= nch;
  const int cg = local % ncg;
  const int hk = local / ncg;
  const int kbeg = c * p.chunk;
  const int kend = min(T, kbeg + p.chunk);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lc = lane & 31, lh = lane >> 5;

  // Page indices of this chunk -> LDS (one round trip before the KV stream).
  const int pg0 = kbeg / kPageSize;
  const int npg = (kend + kPageSize - 1) / kPageSize - pg0;
  for (int i = tid; i < npg; i += kAttnThreads) lds_pages[i] = a.page_indices[rq.page_start + pg0 + i];

  // Query columns of this wave: col = token * g + head-in-group.
  bf16x8 qf[QTW][KSTEPS];
  int lim[QTW];
  bool tile_on[QTW];
  int wave_min_lim = kend;
  for (int qt = 0; qt < QTW; ++qt) {
    const int col0 = cg * cols_per_group + (wave + 4 * qt) * 32;
    tile_on[qt] = col0 < M;
    const int col = col0 + lc;
    const bool valid = col < M;
    const int tok = valid ? col / g : 0;
    const int hh = col - tok * g;
    lim[qt] = valid ? min(kend, tok < nver ? L + tok + 1 : T) : 0;
    if (valid) wave_min_lim = min(wave_min_lim, lim[qt]);
    const uint16_t* qrow = a.q + ((size_t)(rq.q_start + tok) * a.hq + hk * g + hh) * D;
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (valid) w = *(const u32x4*)(qrow + s * 16 + 8 * lh);
      qf[qt][s] = __builtin_bit_cast(bf16x8, w);
    }
  }
  // Smallest visibility limit over the wave's valid columns (wave-uniform).
  for (int off = 32; off >= 1; off >>= 1) wave_min_lim = min(wave_min_lim, __shfl_xor(wave_min_lim, off));

  f32x16 acc[QTW][DT];
  float m_run[QTW], l_run[QTW];
  for (int qt = 0; qt < QTW; ++qt) {
    m_run[qt] = kNegInf;
    l_run[qt] = 0.f;
    for (int dt = 0; dt < DT; ++dt)
      for (int i = 0; i < 16; ++i) acc[qt][dt][i] = 0.f;
  }

  __syncthreads();  // lds_pages ready

  u32x4 kst[PER_THREAD], vst[PER_THREAD];
  const size_t head_stride = (size_t)kPageSize * D;  // elements per (page, head)

  auto load_tile = [&](int k0) {
#pragma unroll
    for (int u = 0; u < PER_THREAD; ++u) {
      const int id = u * kAttnThreads + tid;
      // K: chunk id -> key kk, 16-byte chunk ch of that key's row
      {
        const int kk = id / NCH, ch = id % NCH;
        const int key = k0 + kk;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (key < kend) {
          const int page = lds_pages[key / kPageSize - pg0];
          const uint16_t* src = a.k_cache + ((size_t)page * a.hkv + hk) * head_stride +
                                (size_t)(key % kPageSize) * D + ch * 8;
          w = *(const u32x4*)src;
        }
        kst[u] = w;
      }
      // V: chunk id -> page pp of the tile, head dim d, half (keys 8*half..+7)
      {
        const int pp = id / (2 * D), rem = id % (2 * D);
        const int d = rem >> 1, half = rem & 1;
        const int key = k0 + pp * kPageSize + half * 8;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (key < kend) {
          const int page = lds_pages[key / kPageSize - pg0];
          const uint16_t* src = a.v_cache + ((size_t)page * a.hkv + hk) * head_stride +
                                (size_t)d * kPageSize + half * 8;
          w = *(const u32x4*)src;
          const int valid = kend - key;  // keys of this 8-key run inside the chunk
          if (valid < 8) {
            for (int e = 0; e < 4; ++e) {
              const int k2 = 2 * e;
              uint32_t keep = (k2 < valid ? 0x0000ffffu : 0u) | (k2 + 1 < valid ? 0xffff0000u : 0u);
              w[e] &= keep;
            }
          }
        }
        vst[u] = w;
      }
    }
  };

  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < PER_THREAD; ++u) {
      const int id = u * kAttnThreads + tid;
      {
        const int kk = id / NCH, ch = id % NCH;
        const int phys = ch ^ (swap23(kk & 31) & (NCH - 1));
        *(u32x4*)(&lds_k[buf][kk * D + phys * 8]) = kst[u];
      }
      {
        const int pp = id / (2 * D), rem = id % (2 * D);
        const int d = rem >> 1, half = rem & 1;
        *(u32x4*)(&lds_v[buf][pp * (D * kPageSize) + d * kPageSize + ((half ^ vswz(d)) * 8)]) = vst[u];
      }
    }
  };

  const int ntiles = (kend - kbeg + kKeyTile - 1) / kKeyTile;
  load_tile(kbeg);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int k0 = kbeg + t * kKeyTile;
    const int buf = t & 1;
    if (t + 1 < ntiles) load_tile(k0 + kKeyTile);

    const bool need_mask = k0 + kKeyTile > wave_min_lim;
    f32x16 s[QTW][2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      for (int qt = 0; qt < QTW; ++qt)
        for (int i = 0; i < 16; ++i) s[qt][st][i] = 0.f;
      const int krow = 32 * st + swap23(lc);
      const uint16_t* kbase = &lds_k[buf][krow * D];
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        const int phys = (2 * ks + lh) ^ (lc & (NCH - 1));
        const bf16x8 kf = *(const bf16x8*)(kbase + phys * 8);
        for (int qt = 0; qt < QTW; ++qt)
          if (tile_on[qt]) s[qt][st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qt][ks], s[qt][st], 0, 0, 0);
      }
    }

#pragma unroll
    for (int qt = 0; qt < QTW; ++qt) {
      if (!tile_on[qt]) continue;
      if (need_mask) {
        for (int st = 0; st < 2; ++st)
          for (int i = 0; i < 16; ++i) {
            const int key = k0 + 32 * st + 16 * (i >> 3) + 8 * lh + 4 * ((i >> 2) & 1) + (i & 3);
            if (key >= lim[qt]) s[qt][st][i] = kNegInf;
          }
      }
      float mx = kNegInf;
      for (int st = 0; st < 2; ++st)
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[qt][st][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[qt], mx);
      const bool grew = m_new > m_run[qt];
      if (__any(grew)) {
        const float alpha = grew ? __builtin_amdgcn_exp2f((m_run[qt] - m_new) * a.scale_log2) : 1.f;
        l_run[qt] *= alpha;
        for (int dt = 0; dt < DT; ++dt)
          for (int i = 0; i < 16; ++i) acc[qt][dt][i] *= alpha;
        m_run[qt] = m_new;
      }
      const float mc = (m_new == kNegInf) ? 0.f : m_new * a.scale_log2;
      float lsum = 0.f;
      u32x4 pk[2][2];
      for (int st = 0; st < 2; ++st) {
        float pv[16];
        for (int i = 0; i < 16; ++i) {
          pv[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[qt][st][i], a.scale_log2, -mc));
          lsum += pv[i];
        }
        for (int pp = 0; pp < 2; ++pp)
          for (int e = 0; e < 4; ++e) pk[st][pp][e] = pack_bf16x2(pv[8 * pp + 2 * e], pv[8 * pp + 2 * e + 1]);
      }
      l_run[qt] += lsum;
      // O^T += V^T P^T over the two 32-key sub-tiles (two 16-key MFMA steps each)
      for (int st = 0; st < 2; ++st)
        for (int pp = 0; pp < 2; ++pp) {
          const bf16x8 pf = __builtin_bit_cast(bf16x8, pk[st][pp]);
          const uint16_t* vpage = &lds_v[buf][(2 * st + pp) * (D * kPageSize)];
          for (int dt = 0; dt < DT; ++dt) {
            const int d = 32 * dt + lc;
            const bf16x8 vf = *(const bf16x8*)(vpage + d * kPageSize + ((lh ^ vswz(d)) * 8));
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, acc[qt][dt], 0, 0, 0);
          }
        }
    }

    if (t + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: per column, combine the two half-wave sums.
#pragma unroll
  for (int qt = 0; qt < QTW; ++qt) {
    if (!tile_on[qt]) continue;
    const float l_tot = l_run[qt] + __shfl_xor(l_run[qt], 32);
    const int col = cg * cols_per_group + (wave + 4 * qt) * 32 + lc;
    if (col >= M) continue;
    const int tok = col / g;
    const int hh = col - tok * g;
    const size_t orow = (size_t)(rq.q_start + tok) * a.hq + hk * g + hh;
    if (nch == 1) {
      const float inv = 1.f / l_tot;
      uint16_t* dst = a.out + orow * D;
      for (int dt = 0; dt < DT; ++dt)
        for (int ib = 0; ib < 4; ++ib) {
          u32x2 w;
          w[0] = pack_bf16x2(acc[qt][dt][4 * ib + 0] * inv, acc[qt][dt][4 * ib + 1] * inv);
          w[1] = pack_bf16x2(acc[qt][dt][4 * ib + 2] * inv, acc[qt][dt][4 * ib + 3] * inv);
          *(u32x2*)(dst + 32 * dt + 8 * ib + 4 * lh) = w;
        }
      if (a.lse != nullptr && lh == 0) a.lse[orow] = m_run[qt] * a.sm_scale + __logf(l_tot);
    } else {
      const size_t pcol = (size_t)rq.part_start + ((size_t)hk * nch + c) * M + col;
      float* dst = a.part_o + pcol * D;
      for (int dt = 0; dt < DT; ++dt)
        for (int ib = 0; ib < 4; ++ib) {
          float4 w = make_float4(acc[qt][dt][4 * ib + 0], acc[qt][dt][4 * ib + 1],
                                 acc[qt][dt][4 * ib + 2], acc[qt][dt][4 * ib + 3]);
          *(float4*)(dst + 32 * dt + 8 * ib + 4 * lh) = w;
        }
      if (lh == 0) *(float2*)(a.part_ml + 2 * pcol) = make_float2(m_run[qt], l_tot);
    }
  }
}

// Merge of the split-KV partials: 4 columns per work group, 64 threads per
// column, D/64 head dims per thread.
template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a, AttnPlan p) {
  constexpr int PER = D / 64;
  const int item = xcd_item(p.grid_comb);
  if (item >= p.total_comb) return;
  const int r = find_request(p, item, true);
  const AttnReq rq = p.req[r];
  const int n = rq.nv & 0xffff, L = rq.ctx, T = L + n;
  const int g = a.g;
  const int M = n * g;
  const int nch = (T + p.chunk - 1) / p.chunk;
  const int groups = (M + 3) / 4;
  const int local = item - rq.comb_start;
  const int hk = local / groups;
  const int col = (local % groups) * 4 + (threadIdx.x >> 6);
  if (col >= M) return;
  const int t = threadIdx.x & 63;
  const size_t base = (size_t)rq.part_start + (size_t)hk * nch * M + col;

  float mmax = kNegInf;
  for (int s = 0; s < nch; ++s) mmax = fmaxf(mmax, a.part_ml[2 * (base + (size_t)s * M)]);
  float lsum = 0.f;
  float o[PER];
  for (int e = 0; e < PER; ++e) o[e] = 0.f;
  for (int s = 0; s < nch; ++s) {
    const size_t pc = base + (size_t)s * M;
    const float2 ml = *(const float2*)(a.part_ml + 2 * pc);
    const float w = __builtin_amdgcn_exp2f((ml.x - mmax) * a.scale_log2);
    lsum += w * ml.y;
    const float* src = a.part_o + pc * D + t * PER;
    for (int e = 0; e < PER; ++e) o[e] += w * src[e];
  }
  const int tok = col / g;
  const int hh = col - tok * g;
  const size_t orow = (size_t)(rq.q_start + tok) * a.hq + hk * g + hh;
  const float inv = 1.f / lsum;
  if (PER == 2) {
    *(uint32_t*)(a.out + orow * D + 2 * t) = pack_bf16x2(o[0] * inv, o[1] * inv);
  } else {
    __bf16 b = (__bf16)(o[0] * inv);
    a.out[orow * D + t] = __builtin_bit_cast(uint16_t, b);
  }
  if (a.lse != nullptr && t == 0) a.lse[orow] = mmax * a.sm_scale + __logf(lsum);
}

template <int D, int QTW>
hipError_t launch_impl(const AttnArgs& args, const AttnPlan& plan, hipStream_t stream) {
  hipLaunchKernelGGL((attn_fwd_kernel<D, QTW>), dim3(plan.grid_items), dim3(kAttnThreads), 0, stream,
                     args, plan);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (plan.total_comb > 0) {
    hipLaunchKernelGGL((attn_combine_kernel<D>), dim3(plan.grid_comb), dim3(256), 0, stream, args, plan);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& args, const AttnPlan& plan, int head_dim,
                            hipStream_t stream) {
  const bool wide = plan.cols_per_group > 128;
  if (head_dim == 128) return wide ? launch_impl<128, 2>(args, plan, stream) : launch_impl<128, 1>(args, plan, stream);
  return wide ? launch_impl<64, 2>(args, plan, stream) : launch_impl<64, 1>(args, plan, stream);
}

}  // namespace rg

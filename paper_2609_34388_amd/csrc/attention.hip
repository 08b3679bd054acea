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

// Direct global -> LDS copy of 16 bytes per lane (LDS-DMA).  The wave's 64
// lanes fill 1 KiB of LDS starting at `lds_byte_addr` (lane L at +16 L).
// Issued through inline assembly so that the compiler does not insert a
// wait for every outstanding copy before each LDS read; the kernel waits on
// the vector-memory counter itself.  m0 is saved and restored around it.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_byte_addr) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(__builtin_amdgcn_readfirstlane(lds_byte_addr)), "v"(gptr)
      : "memory");
}

// Wait until at most n vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

constexpr int kStages = 4;  // LDS ring depth (key tiles in flight: kStages - 1)

template <int D, int W>
__global__ __launch_bounds__(64 * W) void attn_fwd_kernel(AttnArgs a, AttnPlan p) {
  constexpr int NT = 64 * W;          // threads
  constexpr int NCH = D / 8;          // 16-byte chunks per K row
  constexpr int KSTEPS = D / 16;      // MFMA k-steps of q.k
  constexpr int DT = D / 32;          // 32-wide head-dim tiles of the output
  constexpr int TILE = kKeyTile * D;  // bf16 elements of one staged K (or V) tile
  constexpr int BLOCKS = TILE * 2 / 1024;  // 1 KiB DMA blocks per K (or V) tile
  constexpr int KPB = 1024 / (2 * D);      // keys per K block
  constexpr int VBPP = D / 32;             // V blocks per page
  constexpr int G = 2 * BLOCKS / W;        // DMA instructions per wave per tile
  constexpr int MAXPAGES = kMaxChunkKeys / kPageSize;
  static_assert(2 * BLOCKS % W == 0, "DMA blocks must split evenly over waves");

  __shared__ __attribute__((aligned(16))) uint16_t lds_k[kStages][TILE];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v[kStages][TILE];
  __shared__ int32_t lds_pages[MAXPAGES];

  const int item = xcd_item(p.grid_items);
  if (item >= p.total_items) return;
  const int r = find_request(p, item, false);
  const AttnReq rq = p.req[r];
  const int n = rq.nv & 0xffff, nver = rq.nv >> 16, L = rq.ctx, T = L + n;
  const int g = a.g;
  const int M = n * g;
  const int cols_per_group = 32 * W;
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

  // This wave's 32 query columns: col = token * g + head-in-group.
  const int col0 = cg * cols_per_group + wave * 32;
  const bool tile_on = col0 < M;  // wave-uniform
  const int col = col0 + lc;
  const bool valid = col < M;
  const int tok = valid ? col / g : 0;
  const int hh = col - tok * g;
  const int lim = valid ? min(kend, tok < nver ? L + tok + 1 : T) : 0;
  bf16x8 qf[KSTEPS];
  {
    const uint16_t* qrow = a.q + ((size_t)(rq.q_start + tok) * a.hq + hk * g + hh) * D;
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (valid) w = *(const u32x4*)(qrow + s * 16 + 8 * lh);
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }
  int wave_min_lim = valid ? lim : kend;
  for (int off = 32; off >= 1; off >>= 1) wave_min_lim = min(wave_min_lim, __shfl_xor(wave_min_lim, off));

  // Page indices of this chunk -> LDS (the one dependent round trip before the KV stream).
  const int pg0 = kbeg / kPageSize;
  const int npg = (kend + kPageSize - 1) / kPageSize - pg0;
  for (int i = tid; i < npg; i += NT) lds_pages[i] = a.page_indices[rq.page_start + pg0 + i];
  __syncthreads();

  const size_t head_stride = (size_t)kPageSize * D;  // elements per (page, head)
  const uint16_t* kbase_g = a.k_cache + (size_t)hk * head_stride;
  const uint16_t* vbase_g = a.v_cache + (size_t)hk * head_stride;
  const size_t page_stride = (size_t)a.hkv * head_stride;
  const int last_key = kend - 1;

  // Issue the DMA of key tile `t` into ring stage t % kStages.  Keys past the
  // chunk end read the chunk's last key (always a valid token); their scores
  // are masked and their values zeroed before use.
  auto issue = [&](int t) {
    const int k0 = kbeg + t * kKeyTile;
    const int st = t % kStages;
    const uint32_t kl = (uint32_t)(uintptr_t)&lds_k[st][0];
    const uint32_t vl = (uint32_t)(uintptr_t)&lds_v[st][0];
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int b = wave + i * W;  // block 0 .. 2*BLOCKS-1 (K blocks first)
      if (b < BLOCKS) {
        const int kk = b * KPB + lane / NCH;
        const int pc = lane % NCH;
        const int ch = pc ^ (swap23(kk & 31) & (NCH - 1));
        const int key = min(k0 + kk, last_key);
        const int page = lds_pages[key / kPageSize - pg0];
        dma16(kbase_g + page * page_stride + (size_t)(key % kPageSize) * D + ch * 8, kl + b * 1024);
      } else {
        const int vb = b - BLOCKS;
        const int pp = vb / VBPP;
        const int d = (vb % VBPP) * 32 + (lane >> 1);
        const int half = (lane & 1) ^ vswz(d);
        const int key = min(k0 + pp * kPageSize, last_key);
        const int page = lds_pages[key / kPageSize - pg0];
        dma16(vbase_g + page * page_stride + (size_t)d * kPageSize + half * 8, vl + vb * 1024);
      }
    }
  };

  f32x16 acc[DT];
  for (int dt = 0; dt < DT; ++dt)
    for (int i = 0; i < 16; ++i) acc[dt][i] = 0.f;
  float m_run = kNegInf, l_run = 0.f;

  const int ntiles = (kend - kbeg + kKeyTile - 1) / kKeyTile;
  for (int t = 0; t < kStages - 1 && t < ntiles; ++t) issue(t);

  for (int t = 0; t < ntiles; ++t) {
    if (t + kStages - 1 < ntiles) issue(t + kStages - 1);
    const int ahead = min(kStages - 1, ntiles - 1 - t);  // tiles issued after tile t
    if (ahead >= 3) wait_vmcnt<3 * G>();
    else if (ahead == 2) wait_vmcnt<2 * G>();
    else if (ahead == 1) wait_vmcnt<G>();
    else wait_vmcnt<0>();
    __syncthreads();

    const int k0 = kbeg + t * kKeyTile;
    const int st = t % kStages;
    const int nvalid = kend - k0;
    if (nvalid < kKeyTile) {
      // last tile of the chunk: zero the values of keys past its end
      for (int i = tid; i < kKeyTile * D; i += NT) {
        const int kk = i / D, d = i % D;
        if (kk >= nvalid) {
          const int pp = kk / kPageSize, kp = kk % kPageSize;
          lds_v[st][pp * (D * kPageSize) + d * kPageSize + (((kp >> 3) ^ vswz(d)) * 8) + (kp & 7)] = 0;
        }
      }
      __syncthreads();
    }

    if (tile_on) {
      const bool need_mask = k0 + kKeyTile > wave_min_lim;
      f32x16 s[2];
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        for (int i = 0; i < 16; ++i) s[sub][i] = 0.f;
        const int krow = 32 * sub + swap23(lc);
        const uint16_t* kb = &lds_k[st][krow * D];
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
          const int phys = (2 * ks + lh) ^ (lc & (NCH - 1));
          const bf16x8 kf = *(const bf16x8*)(kb + phys * 8);
          s[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[sub], 0, 0, 0);
        }
      }
      if (need_mask) {
        for (int sub = 0; sub < 2; ++sub)
          for (int i = 0; i < 16; ++i) {
            const int key = k0 + 32 * sub + 16 * (i >> 3) + 8 * lh + 4 * ((i >> 2) & 1) + (i & 3);
            if (key >= lim) s[sub][i] = kNegInf;
          }
      }
      float mx = kNegInf;
      for (int sub = 0; sub < 2; ++sub)
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[sub][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const bool grew = m_new > m_run;
      if (__any(grew)) {
        const float alpha = grew ? __builtin_amdgcn_exp2f((m_run - m_new) * a.scale_log2) : 1.f;
        l_run *= alpha;
        for (int dt = 0; dt < DT; ++dt)
          for (int i = 0; i < 16; ++i) acc[dt][i] *= alpha;
        m_run = m_new;
      }
      const float mc = (m_new == kNegInf) ? 0.f : m_new * a.scale_log2;
      float lsum = 0.f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        u32x4 pk[2];
        for (int pp = 0; pp < 2; ++pp)
          for (int e = 0; e < 4; ++e) {
            const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[sub][8 * pp + 2 * e], a.scale_log2, -mc));
            const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[sub][8 * pp + 2 * e + 1], a.scale_log2, -mc));
            lsum += p0 + p1;
            pk[pp][e] = pack_bf16x2(p0, p1);
          }
        // O^T += V^T P^T: two 16-key MFMA steps per 32-key sub-tile
        for (int pp = 0; pp < 2; ++pp) {
          const bf16x8 pf = __builtin_bit_cast(bf16x8, pk[pp]);
          const uint16_t* vpage = &lds_v[st][(2 * sub + pp) * (D * kPageSize)];
          for (int dt = 0; dt < DT; ++dt) {
            const int d = 32 * dt + lc;
            const bf16x8 vf = *(const bf16x8*)(vpage + d * kPageSize + ((lh ^ vswz(d)) * 8));
            acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, acc[dt], 0, 0, 0);
          }
        }
      }
      l_run += lsum;
    }
    __syncthreads();  // stage st is refilled by the next iteration's DMA
  }

  // Epilogue: per column, combine the two half-wave sums.
  if (!tile_on || !valid) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const size_t orow = (size_t)(rq.q_start + tok) * a.hq + hk * g + hh;
  if (nch == 1) {
    const float inv = 1.f / l_tot;
    uint16_t* dst = a.out + orow * D;
    for (int dt = 0; dt < DT; ++dt)
      for (int ib = 0; ib < 4; ++ib) {
        u32x2 w;
        w[0] = pack_bf16x2(acc[dt][4 * ib + 0] * inv, acc[dt][4 * ib + 1] * inv);
        w[1] = pack_bf16x2(acc[dt][4 * ib + 2] * inv, acc[dt][4 * ib + 3] * inv);
        *(u32x2*)(dst + 32 * dt + 8 * ib + 4 * lh) = w;
      }
    if (a.lse != nullptr && lh == 0) a.lse[orow] = m_run * a.sm_scale + __logf(l_tot);
  } else {
    const size_t pcol = (size_t)rq.part_start + ((size_t)hk * nch + c) * M + col;
    float* dst = a.part_o + pcol * D;
    for (int dt = 0; dt < DT; ++dt)
      for (int ib = 0; ib < 4; ++ib) {
        float4 w = make_float4(acc[dt][4 * ib + 0], acc[dt][4 * ib + 1], acc[dt][4 * ib + 2], acc[dt][4 * ib + 3]);
        *(float4*)(dst + 32 * dt + 8 * ib + 4 * lh) = w;
      }
    if (lh == 0) *(float2*)(a.part_ml + 2 * pcol) = make_float2(m_run, l_tot);
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

template <int D, int W>
hipError_t launch_impl(const AttnArgs& args, const AttnPlan& plan, hipStream_t stream) {
  hipLaunchKernelGGL((attn_fwd_kernel<D, W>), dim3(plan.grid_items), dim3(64 * W), 0, stream, args, plan);
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
  if (head_dim == 128) return wide ? launch_impl<128, 8>(args, plan, stream) : launch_impl<128, 4>(args, plan, stream);
  return wide ? launch_impl<64, 8>(args, plan, stream) : launch_impl<64, 4>(args, plan, stream);
}

}  // namespace rg

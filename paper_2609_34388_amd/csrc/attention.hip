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
// request that share the KV head -- n * Hq/Hkv of them, up to 256 per group --
// so every K/V byte of a chunk is read from HBM once for all of them.  The 8
// compute waves of a work group split the group into 32-column tiles and,
// when there are fewer than 8 tiles, the chunk's 32-key sub-tiles into key
// groups; 4 more waves only copy K and V into LDS.
// Requests whose keys span several chunks write normalised partial outputs
// plus (max, sum) per column; a second kernel merges them with the usual
// log-sum-exp weights (or, in the opt-in one-launch mode, merge items of the
// same launch, taken from a work queue once the chunks they merge are done).
//
// K and V of 128 keys (8 pages) at a time pass through LDS (two slots each):
// the copy waves load the next two buffers into registers with ordinary
// vector loads while the current one is computed, and write each to its LDS
// slot just before its barrier.  On each 32-key sub-tile a wave forms
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K rows are the MFMA rows, query
// columns the MFMA columns), applies the mask, updates the running max and
// sum in fp32 (exp2 with the scale folded in), converts P to bf16 and
// accumulates O^T += V^T P^T with the same MFMA.  The K rows of a sub-tile are loaded in a
// permuted order (bits 2 and 3 of the row index swapped) so that the S^T
// accumulator registers a lane holds are exactly the P^T operand the PV MFMA
// needs and the matching V^T operand is 8 consecutive keys of one head
// dimension: 16 contiguous bytes of a dimension-major V page.
//
// Bounds: a work group reads only pages of its own chunk (whole pages of the
// pool, unused slots of a request's last page included); buffer rows past
// the chunk end get their scores masked to -inf and their values zeroed, so
// whatever those slots hold (NaN included) never reaches the output.
#include <type_traits>

#include "rg_internal.h"

namespace rg {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ int swap23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Swizzle of the two 16-byte halves of a dimension row of a V page in LDS.
__device__ __forceinline__ int vswz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Request owning work item `item`: the last r with start(r) <= item (starts
// are nondecreasing, empty requests share their successor's start).  Every
// lane tests one request, so the search is one round of loads, not a chain.
template <typename Plan>
__device__ __forceinline__ int find_request(const Plan& p, int item, bool combine) {
  const int lane = threadIdx.x & 63;
  int r = 0;
  for (int base = 1; base < p.num_req; base += 64) {
    const int k = base + lane;
    const bool le = k < p.num_req && (combine ? p.req[k].comb_start : p.req[k].item_start) <= item;
    r += __popcll(__ballot(le));
  }
  return __builtin_amdgcn_readfirstlane(r);
}

// Consecutive work items of one (request, KV head) land on one XCD: the
// dispatcher deals work groups to the 8 XCDs round-robin, so block b runs on
// XCD b % 8; give XCD x the item range [x*per, (x+1)*per).
__device__ __forceinline__ int xcd_item(int grid_items) {
  const int per = grid_items >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

// Work-group barrier that orders LDS only.  __syncthreads() also fences
// global memory, which makes every wave wait for all of its outstanding
// vector-memory operations -- the copy waves' loads of the next buffers --
// at each barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wait until at most n vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Device-coherent stores and loads (agent-scope relaxed atomics: the stores
// write through to the level all XCDs share, the loads read from it), used
// for the split-KV partials that a combine item of the same launch reads,
// possibly on another XCD.  Ordering between a wave's stores and the count it
// publishes afterwards comes from waiting for the stores to complete
// (vmcnt 0) before the counting atomic; the reader's loads are issued only
// after it has seen the full count.  No cache-wide write-back or invalidate
// is needed, because only these locations are shared.
__device__ __forceinline__ void store16_coherent(uint16_t* p, u32x4 w) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  __hip_atomic_store(q, (uint64_t)w[0] | ((uint64_t)w[1] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, (uint64_t)w[2] | ((uint64_t)w[3] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store8_coherent(float* p, float x, float y) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p),
                     (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ u32x4 load16_coherent(const uint16_t* p) {
  const uint64_t* q = reinterpret_cast<const uint64_t*>(p);
  const uint64_t lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return u32x4{(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)};
}
__device__ __forceinline__ float2 load8_coherent(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

constexpr int kWaves = 8;      // compute waves per work group (two per SIMD)
constexpr int kProducers = 4;  // copy waves per work group (one per SIMD)
constexpr int kThreads = 64 * (kWaves + kProducers);
constexpr int kSuper = 128;  // keys staged per LDS buffer (four 32-key sub-tiles)
constexpr int kKBufs = 2;    // K buffers: one computed, one being filled
constexpr int kVBufs = 2;    // V buffers: one computed, one being filled
static_assert(kKBufs == 2 && kVBufs == 2, "two copy-wave pairs, one per buffer parity and LDS slot");
static_assert(kSuper % kKeyTile == 0, "a super-tile is a whole number of key tiles");

// Work group = 8 compute waves over (column tiles) x (key groups).  A
// request's columns are split into groups of up to 256 (8 tiles of 32); a
// wave handling key group kgi of kg processes the chunk's 32-key sub-tiles j
// with j % kg == kgi.  Small requests thus keep all 8 waves (two per SIMD)
// busy on disjoint keys; the key groups' partial softmax states are merged
// through LDS at the end.
//
// Keys stream through LDS 128 at a time (K and V of 8 pages), one barrier per
// 128 keys.  The copies are made by 4 dedicated waves (one per SIMD), two per
// buffer parity, each holding its share of a buffer (32 KiB per pair) in
// registers from its load until just before that buffer's barrier: two
// buffers are in flight from HBM, and the compute waves spend no issue slots
// or registers on copies.  (Loads straight into LDS, which need no staging
// registers, measured slower: a CU takes such a 1 KiB load only every few
// dozen cycles, about 5.9 TB/s over the chip against about 7.1 TB/s for
// plain vector loads.)
//
// PERSIST: the item runs inside the one-launch work-queue kernel.  Every wave
// then passes the same barriers (the copy waves join the key-group merge),
// and a split item's partials are stored device-coherently and counted so
// that the combine items of the same launch can merge them.
template <int D, typename Plan, bool PERSIST>
__device__ __forceinline__ void attn_item(const AttnArgs& a, const Plan& p, const int item, uint16_t* lds) {
  constexpr bool BR = __is_same(Plan, AttnPlanBr);  // rows after the verify rows form branches
  constexpr int NCH = D / 8;                   // 16-byte chunks per K row
  constexpr int KSTEPS = D / 16;               // MFMA k-steps of q.k
  constexpr int DT = D / 32;                   // 32-wide head-dim tiles of the output
  constexpr int SUPER = kSuper * D;            // bf16 elements of one K (or V) buffer
  constexpr int BLOCKS = SUPER * 2 / 1024;     // 1 KiB copy blocks per K (or V) buffer
  constexpr int KPB = 1024 / (2 * D);          // keys per K block
  constexpr int VBPP = D / 32;                 // V blocks per page
  constexpr int COLS = 32 * kWaves;            // columns per column group
  // key-group merge: one slot per wave that hands its state over (every such wave has index >= 1)
  static_assert((kKBufs + kVBufs) * SUPER * 2 >= (kWaves - 1) * (64 * 16 * DT + 128) * 4, "merge area");

  // kbuf[b] = K of 128 keys ([key][D], 16-byte chunks swizzled per row),
  // vbuf[b] = V of 8 pages ([page][D][16 keys], halves swizzled per row).
  // Two slots of each (128 KiB of LDS at D = 128): buffer s in slot s % 2
  // while buffer s + 1 is written into the other.
  auto kbuf = [&](int s) { return lds + (s % kKBufs) * SUPER; };
  auto vbuf = [&](int s) { return lds + (kKBufs + s % kVBufs) * SUPER; };

  const int r = find_request(p, item, false);
  const auto rq = p.req[r];
  // both counts are 16-bit fields of one word: unpack unsigned (n_verify may reach 65535)
  const int n = rq.nv & 0xffff, nver = (int)((uint32_t)rq.nv >> 16), L = rq.ctx, T = L + n;
  const int g = a.g;
  const int M = n * g;
  const int ncg = (M + COLS - 1) / COLS;
  // The request's 32-column tiles are dealt evenly to its column groups
  // (e.g. 17 tiles as 6, 6, 5 rather than 8, 8, 1), so the groups, which
  // read the same keys, run at about the same pace.
  const int tpg = ((M + 31) / 32 + ncg - 1) / ncg;
  const int nch = (T + p.chunk - 1) / p.chunk;
  // A request's items run over chunks, then KV heads, then column groups:
  // the items of one (KV head, chunk) for successive column groups lie
  // Hkv * chunks apart -- with 8 KV heads, 8 apart, so on the same XCD
  // (work group b runs on XCD b % 8; every request's items start at a
  // multiple of 8 then) and dispatched together, and the column groups after
  // the first mostly find the keys in that XCD's L2 instead of HBM.
  int local = item - rq.item_start;
  const int c = local % nch;
  local /= nch;
  const int hk = local % a.hkv;
  const int cg = local / a.hkv;
  const int kbeg = c * p.chunk;
  const int kend = min(T, kbeg + p.chunk);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, in an SGPR
  const int lc = lane & 31, lh = lane >> 5;

  // Column tiles of this group and each compute wave's (column tile ct, key
  // group kgi of kg; the tile's other key groups are waves w + k kstride).
  // Compute waves w and w + 4 share a SIMD.  Up to 4 tiles: every tile gets
  // 8 / nct' waves (nct' = nct rounded up to a power of two).  5 to 7 tiles:
  // tiles 0-3 get waves 0-3 and the rest share waves 4-7 by key groups, so
  // no SIMD carries two whole tiles while another idles.
  const int nct = min(tpg, (M + 31) / 32 - cg * tpg);
  const bool producer = wave >= kWaves;  // wave-uniform: copy wave
  // Pages of this chunk: entries pg0 .. pg0 + npg - 1 of the request's list.
  const int pg0 = kbeg / kPageSize;
  const int npg = (kend + kPageSize - 1) / kPageSize - pg0;
  // The copy waves read page numbers through the scalar cache (uniform
  // addresses in the constant address space): no LDS stage, no barrier.
  typedef const int32_t __attribute__((address_space(4))) * cpage_ptr;
  const cpage_ptr chunk_pages = (cpage_ptr)(a.page_indices + rq.page_start + pg0);

  const size_t head_stride = (size_t)kPageSize * D;  // elements per (page, head)
  const char* kbase_g = reinterpret_cast<const char*>(a.k_cache + (size_t)hk * head_stride);
  const char* vbase_g = reinterpret_cast<const char*>(a.v_cache + (size_t)hk * head_stride);
  const size_t page_bytes = (size_t)a.hkv * head_stride * 2;

  // Copy waves.  The four copy waves form two pairs, one per buffer parity:
  // pair `par` copies buffers par, par + 2, ... into LDS slot par.  Wave q of
  // the pair moves K blocks b = q + 2 i and V blocks b = q + 2 i of its
  // buffer (i = 0 .. NB - 1): a K block is KPB keys, a V block 32 head dims of
  // one page, 1 KiB each; lane L's 16 bytes of a block go to byte 16 L of the
  // block's place in the slot.  A wave reads its buffer's 8 page numbers
  // (one batch of scalar loads), loads its blocks into registers and writes
  // them to LDS before the buffer's barrier.  Page slots past the chunk's
  // last page repeat that page, so buffer rows past the chunk end hold other
  // tokens or unused slots of the last page (memory of the pool either way);
  // their scores are masked and their values zeroed before use.
  constexpr int WPG = kProducers / 2;  // copy waves per parity
  constexpr int NB = BLOCKS / WPG;     // K (and V) blocks per copy wave and buffer
  static_assert(BLOCKS % WPG == 0 && NB % 2 == 0, "blocks split evenly over a pair");
  const int pw = wave - kWaves;
  const int par = pw / WPG;  // wave-uniform: buffer parity (and LDS slot) of this copy wave
  const int q = pw % WPG;
  // A buffer's 8 page numbers: one 32-byte scalar load when all 8 are the
  // chunk's (else one load per slot, repeating the last page), so the copies
  // wait for one scalar round trip, not eight.
  typedef int32_t i32x8 __attribute__((ext_vector_type(8), aligned(4)));
  typedef const i32x8 __attribute__((address_space(4))) * cpage8_ptr;
  static_assert(kSuper / kPageSize == 8, "eight pages per buffer");
  auto read_pages = [&](int s, int (&pg)[kSuper / kPageSize]) {
    const int base = s * (kSuper / kPageSize);
    if (base + 8 <= npg) {
      const i32x8 v = *(cpage8_ptr)(chunk_pages + base);
#pragma unroll
      for (int j = 0; j < 8; ++j) pg[j] = v[j];
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) pg[j] = chunk_pages[min(base + j, npg - 1)];
    }
  };
  // A lane's byte offset inside its page repeats with period 2 in i: blocks
  // i and i + 2 lie 2 WPG = 4 blocks apart, 4 KPB keys (a multiple of 16,
  // so the same page slot and the same swap23 row bits) or 4 V blocks (a
  // multiple of VBPP, so the same head dims).
  static_assert((2 * WPG * KPB) % kPageSize == 0 && (2 * WPG) % VBPP == 0, "offsets repeat every two blocks");
  uint32_t koff[2], voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int b = q + WPG * e;
    const int kk = b * KPB + lane / NCH;
    koff[e] = (uint32_t)((((kk % kPageSize) * D) + (((lane % NCH) ^ (swap23(kk & 31) & (NCH - 1))) * 8)) * 2);
    const int d = (b % VBPP) * 32 + (lane >> 1);
    voff[e] = (uint32_t)((d * kPageSize + ((lane & 1) ^ vswz(d)) * 8) * 2);
  }
  // This wave's blocks of one buffer: NB K blocks, then NB V blocks.
  auto load_set = [&](const int (&pg)[kSuper / kPageSize], u32x4 (&r)[2 * NB]) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = q + WPG * i;
      r[i] = __builtin_nontemporal_load(
          (const u32x4*)(kbase_g + (size_t)pg[(b * KPB) / kPageSize] * page_bytes + koff[i & 1]));
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = q + WPG * i;
      r[NB + i] = __builtin_nontemporal_load((const u32x4*)(vbase_g + (size_t)pg[b / VBPP] * page_bytes + voff[i & 1]));
    }
  };
  auto store_set = [&](const u32x4 (&r)[2 * NB]) {
    uint16_t* kd = lds + par * SUPER + q * 512 + lane * 8;
    uint16_t* vd = lds + (kKBufs + par) * SUPER + q * 512 + lane * 8;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      *(u32x4*)(kd + i * WPG * 512) = r[i];
      *(u32x4*)(vd + i * WPG * 512) = r[NB + i];
    }
  };

  const int nsup = (kend - kbeg + kSuper - 1) / kSuper;
  // Zero the values of keys past the chunk end in the last buffer (every
  // wave takes part, so both loops below pass the same barriers), by 16-byte
  // units (page slot pp, head dim d, half h = keys 16 pp + 8 h ..).
  auto tail_fixup = [&](int s, int nvalid) {
    uint16_t* vz = vbuf(s);
    for (int u = tid; u < (kSuper / kPageSize) * D * 2; u += kThreads) {
      const int pp = u / (2 * D), d = (u >> 1) % D, h = u & 1;
      const int kfirst = kPageSize * pp + 8 * h;
      if (kfirst + 8 <= nvalid) continue;
      uint16_t* unit = vz + pp * (D * kPageSize) + d * kPageSize + ((h ^ vswz(d)) * 8);
      if (kfirst >= nvalid) {
        *(u32x4*)unit = u32x4{0u, 0u, 0u, 0u};
      } else {
        for (int e = nvalid - kfirst; e < 8; ++e) unit[e] = 0;
      }
    }
    lds_barrier();
  };

  if (producer) {
    // Buffer s's loads go out after barrier s - 2 (buffers 0 and 1 at the
    // start) and land in LDS slot s % 2 before barrier s -- over buffer
    // s - 2, computed before barrier s - 1 -- so two buffers are in flight
    // per work group, one per pair, and each wave waits only for its own.
    // A pair reads the page numbers of its next buffer right after issuing
    // the loads of the current one, so they are in registers when needed.
    u32x4 r[2 * NB];
    int pg[kSuper / kPageSize];
    if (par < nsup) {
      read_pages(par, pg);
      load_set(pg, r);
      if (par + 2 < nsup) read_pages(par + 2, pg);
    }
    for (int s = 0; s < nsup; ++s) {
      const bool mine = (s & 1) == par;
      if (mine) store_set(r);
      lds_barrier();  // everyone's copies of buffer s are in; buffers of s - 1 are no longer read
      const int nvalid = kend - (kbeg + s * kSuper);
      if (nvalid < kSuper) tail_fixup(s, nvalid);
      if (mine && s + 2 < nsup) {
        load_set(pg, r);  // buffer s + 2, whose page numbers were fetched a round earlier
        if (s + 4 < nsup) read_pages(s + 4, pg);
      }
    }
    if constexpr (PERSIST) {
      if (nct < 8) {  // the key-group merge's two barriers
        lds_barrier();
        lds_barrier();
      }
    }
    return;
  }
  int ct, kg, kgi, kstride;
  if (nct <= 4) {
    const int nct2 = nct <= 1 ? 1 : nct <= 2 ? 2 : 4;
    ct = wave % nct2;
    kg = kWaves / nct2;
    kgi = wave / nct2;
    kstride = nct2;
  } else if (wave < 4 || nct == 8) {
    ct = wave;
    kg = 1;
    kgi = 0;
    kstride = 1;
  } else if (nct == 7) {  // tiles 4, 5 on waves 4, 5; tile 6 on waves 6, 7
    ct = min(wave, 6);
    kg = wave < 6 ? 1 : 2;
    kgi = wave < 6 ? 0 : wave - 6;
    kstride = 1;
  } else {  // 5 tiles: tile 4 on waves 4-7; 6 tiles: tile 4 on 4, 5 and tile 5 on 6, 7
    kg = 4 / (nct - 4);
    ct = 4 + (wave - 4) / kg;
    kgi = (wave - 4) % kg;
    kstride = 1;
  }
  const bool tile_on = !producer && ct < nct;  // wave-uniform
  const int col = (cg * tpg + ct) * 32 + lc;
  const bool valid = tile_on && col < M;
  const int tok = valid ? col / g : 0;
  const int hh = col - tok * g;
  // Keys a column sees: those below lim, and with overlap branches also its
  // branch's own rows slo .. shi - 1 (Eq. 1 on the branch's sequence: the
  // kept canonical prefix, then the branch's committed lead rows causally,
  // then its draft rows seeing the whole branch).  Both clipped to the chunk.
  int lim, slo = 0, shi = 0;
  if (!valid) {
    lim = 0;
  } else if (!BR || tok < nver) {
    lim = min(kend, tok < nver ? L + tok + 1 : T);
  } else {
    int t = tok - nver, start = L + nver, prefix = nver, lead = 0, rows = n - nver;
    if constexpr (BR) {
      // Word `last` stands for `cnt` branches of its shape whose prefixes
      // grow by `stp`; the words before it for one branch each.
      const int cnt = rq.rep & 0xffff, stp = (rq.rep >> 16) & 0xfff, last = (int)((uint32_t)rq.rep >> 28);
      bool found = false;
#pragma unroll
      for (int bb = 0; bb < 3; ++bb) {
        const int w = rq.br[bb];
        const int rb = w & 0xffff;
        if (w != 0 && !found) {
          const int span = bb == last ? rb * cnt : rb;
          if (t < span) {
            const int k = bb == last ? t / rb : 0;
            t -= k * rb;
            start += k * rb;
            prefix = ((w >> 16) & 0xfff) + k * stp;
            lead = (int)((uint32_t)w >> 28);
            rows = rb;
            found = true;
          } else {
            t -= span;
            start += span;
          }
        }
      }
    }
    lim = min(kend, L + prefix);
    slo = start;
    // empty (shi = slo) when the chunk ends before the branch's rows begin
    shi = max(slo, min(kend, start + (t < lead ? t + 1 : rows)));
  }
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

  f32x16 acc[DT];
  for (int dt = 0; dt < DT; ++dt)
    for (int i = 0; i < 16; ++i) acc[dt][i] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // Byte offset of this lane's K fragment ks inside a 32-key sub-tile: row
  // swap23(lc), 16-byte chunk (2 ks + lh) ^ (lc % NCH) = 2 (ks ^ kw) + kb.
  const int kx = lc & (NCH - 1), kw = kx >> 1;
  const uint32_t krow = (uint32_t)(swap23(lc) * D * 2 + ((lh ^ (kx & 1)) * 16));

  // S^T of sub-tile q (keys 32 q .. 32 q + 31 of the buffer).
  auto qk = [&](const uint16_t* kt, int q) {
    const char* kb = reinterpret_cast<const char*>(kt + 32 * q * D);
    bf16x8 kf[KSTEPS];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) kf[ks] = *(const bf16x8*)(kb + krow + ((ks ^ kw) << 5));
    f32x16 sc;
    for (int i = 0; i < 16; ++i) sc[i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], qf[ks], sc, 0, 0, 0);
    return sc;
  };
  // Online softmax of one sub-tile's scores (keys kbase ..): mask, running max
  // (both half-waves of a column agree through a permlane swap), lazy rescale
  // of the accumulator, then O^T += V^T P^T with P rounded to bf16; the
  // running sum adds the same rounded P the MFMA uses.
  auto softmax_pv = [&](f32x16 sc, int kbase, const uint16_t* vt, int q) {
    if (kbase + 32 > wave_min_lim) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kbase + 16 * (i >> 3) + 8 * lh + 4 * ((i >> 2) & 1) + (i & 3);
        if (key >= lim && (!BR || (uint32_t)(key - slo) >= (uint32_t)(shi - slo))) sc[i] = kNegInf;
      }
    }
    float mx = sc[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) mx = fmaxf(mx, sc[i]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    // The reference maximum only moves when a score exceeds it by more than
    // 2^8 in probability: P stays below 256 (exact enough in bf16, far from
    // overflow in fp32) and the accumulator is rescaled rarely.
    const bool grew = mx > m_run + a.rescale_gap;
    if (__any(grew)) {
      const float m_new = grew ? mx : m_run;
      const float alpha = grew ? __builtin_amdgcn_exp2f((m_run - m_new) * a.scale_log2) : 1.f;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[dt][i] *= alpha;
      m_run = m_new;
    }
    const float mc = (m_run == kNegInf) ? 0.f : m_run * a.scale_log2;
    u32x4 pk[2];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const f32x2 pr = {__builtin_amdgcn_exp2f(__builtin_fmaf(sc[8 * pp + 2 * e], a.scale_log2, -mc)),
                          __builtin_amdgcn_exp2f(__builtin_fmaf(sc[8 * pp + 2 * e + 1], a.scale_log2, -mc))};
        const bf16x2 pb = __builtin_convertvector(pr, bf16x2);
        l_run = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, l_run, false);
        pk[pp][e] = __builtin_bit_cast(uint32_t, pb);
      }
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      bf16x8 vf[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d = 32 * dt + lc;
        vf[dt] = *(const bf16x8*)(vt + (2 * q + pp) * (D * kPageSize) + d * kPageSize + ((lh ^ vswz(d)) * 8));
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[dt], __builtin_bit_cast(bf16x8, pk[pp]), acc[dt], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the next sub-tile's loads after this one's PV
  };
  for (int s = 0; s < nsup; ++s) {
    lds_barrier();
    const int k0 = kbeg + s * kSuper;
    const int nvalid = kend - k0;
    if (nvalid < kSuper) tail_fixup(s, nvalid);
    if (tile_on) {
      const uint16_t* kt = kbuf(s);
      const uint16_t* vt = vbuf(s);
      // this wave's sub-tiles of the buffer: global sub-tile j = 4 s + q with j % kg == kgi
      for (int q = 0; q < kSuper / 32; ++q)
        if (((4 * s + q) & (kg - 1)) == kgi && 32 * q < nvalid) softmax_pv(qk(kt, q), k0 + 32 * q, vt, q);
    }
  }


  // Merge the key groups' partial states (lane-wise: same columns, same dims).
  // A wave's slot holds its accumulator as 16-byte rows, lane-interleaved.
  float l_tot = l_run + __shfl_xor(l_run, 32);
  if (nct < 8) {  // some tile is split over key groups (uniform: every compute wave passes the barriers)
    lds_barrier();  // every wave is done with the buffers before they are reused
    float* area = reinterpret_cast<float*>(lds);
    constexpr int PER = 64 * 16 * DT + 128;  // floats per wave slot
    if (tile_on && kgi > 0) {
      float* slot = area + (wave - 1) * PER;
      for (int dt = 0; dt < DT; ++dt)
        for (int ib = 0; ib < 4; ++ib)
          *(float4*)(slot + ((dt * 4 + ib) * 64 + lane) * 4) =
              make_float4(acc[dt][4 * ib], acc[dt][4 * ib + 1], acc[dt][4 * ib + 2], acc[dt][4 * ib + 3]);
      slot[64 * 16 * DT + lane] = m_run;
      slot[64 * 16 * DT + 64 + lane] = l_tot;
    }
    lds_barrier();
    if (!tile_on || kgi > 0) return;
    for (int k = 1; k < kg; ++k) {
      const float* slot = area + (wave + k * kstride - 1) * PER;
      const float mk = slot[64 * 16 * DT + lane];
      if (mk == kNegInf) continue;
      const float lk = slot[64 * 16 * DT + 64 + lane];
      const float m_new = fmaxf(m_run, mk);
      const float a0 = __builtin_amdgcn_exp2f((m_run - m_new) * a.scale_log2);
      const float a1 = __builtin_amdgcn_exp2f((mk - m_new) * a.scale_log2);
      for (int dt = 0; dt < DT; ++dt)
        for (int ib = 0; ib < 4; ++ib) {
          const float4 o = *(const float4*)(slot + ((dt * 4 + ib) * 64 + lane) * 4);
          acc[dt][4 * ib] = acc[dt][4 * ib] * a0 + o.x * a1;
          acc[dt][4 * ib + 1] = acc[dt][4 * ib + 1] * a0 + o.y * a1;
          acc[dt][4 * ib + 2] = acc[dt][4 * ib + 2] * a0 + o.z * a1;
          acc[dt][4 * ib + 3] = acc[dt][4 * ib + 3] * a0 + o.w * a1;
        }
      l_tot = l_tot * a0 + lk * a1;
      m_run = m_new;
    }
  }

  // Epilogue.
  if (nch == 1) {
    if (!valid) return;
    const size_t orow = (size_t)(rq.q_start + tok) * a.hq + hk * g + hh;
    const float inv = 1.f / l_tot;
    uint16_t* dst = a.out + orow * D;
    for (int dt = 0; dt < DT; ++dt)
      for (int ib = 0; ib < 4; ++ib) {
        const f32x2 lo = {acc[dt][4 * ib + 0] * inv, acc[dt][4 * ib + 1] * inv};
        const f32x2 hi = {acc[dt][4 * ib + 2] * inv, acc[dt][4 * ib + 3] * inv};
        u32x2 w;
        w[0] = __builtin_bit_cast(uint32_t, __builtin_convertvector(lo, bf16x2));
        w[1] = __builtin_bit_cast(uint32_t, __builtin_convertvector(hi, bf16x2));
        *(u32x2*)(dst + 32 * dt + 8 * ib + 4 * lh) = w;
      }
    if (a.lse != nullptr && lh == 0) a.lse[orow] = m_run * a.sm_scale + __logf(l_tot);
  } else {
    // Partial of this 32-column tile: the chunk's normalised output o / l in
    // bf16 (with its fp32 max and sum beside it), stored in the accumulator's
    // own order: 16-byte row (dt, j) of lane l (its registers 8 j .. 8 j + 7)
    // at ((dt * 2 + j) * 64 + l) * 16 bytes, so every store instruction writes
    // 1 KiB contiguously.
    // In the one-launch kernel the stores are device-coherent (they reach
    // the point every XCD reads from before the wave's wait below ends), and
    // then the wave adds its tile to the column group's finished count.
    const int M32 = (M + 31) & ~31;
    const size_t tile0 = (size_t)rq.part_start + ((size_t)hk * nch + c) * M32 + (size_t)((cg * tpg + ct) * 32);
    uint16_t* dst = a.part_o + tile0 * D;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;  // 0: no key of this chunk is visible to the column
    if (valid) {
      for (int dt = 0; dt < DT; ++dt)
        for (int j = 0; j < 2; ++j) {
          u32x4 w;
          for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(acc[dt][8 * j + 2 * e] * inv, acc[dt][8 * j + 2 * e + 1] * inv);
          uint16_t* at = dst + ((dt * 2 + j) * 64 + lane) * 8;
          if constexpr (PERSIST) store16_coherent(at, w);
          else *(u32x4*)at = w;
        }
      if (lh == 0) {
        if constexpr (PERSIST) store8_coherent(a.part_ml + 2 * (tile0 + lc), m_run, l_tot);
        else *(float2*)(a.part_ml + 2 * (tile0 + lc)) = make_float2(m_run, l_tot);
      }
    }
    if constexpr (PERSIST) {
      wait_vmcnt<0>();
      if (lane == 0)
        __hip_atomic_fetch_add(a.sync + kSyncHeader + rq.comb_start + hk * ncg + cg, 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Merge of the split-KV partials.  Work item = (request, KV head, 32-column
// tile, slice of ROWS 16-byte rows of the tile's fragment-ordered block).  A
// row (8 head dims of one column: two runs of 4) is merged by PARTS threads:
// part j takes chunks j, j + PARTS, ... -- up to eight chunks' loads in
// flight at a time -- and merges them with online rescaling (chunk weight
// exp(m_c - m) * l_c on the chunk's normalised output); the parts' states
// then meet in LDS (`st`, (PARTS - 1) x 10 x ROWS floats) and part 0 merges
// them in order and writes 8 bf16 outputs.
//
// PERSIST: the item is a combine item of the one-launch kernel.  Thread 0
// first waits until every tile of every chunk of the item's column group has
// been counted finished (all of those main items were taken from the queue
// before any combine item, by running work groups, so the wait ends; a
// bounded spin sets the error word instead of hanging if it ever did not),
// and the partials are read device-coherently.  The last combine item of a
// column group to pass the wait returns its two counters to zero for the
// next call.
constexpr int kCombRows = 128;         // 16-byte rows per item of the combine kernel
constexpr int kCombRowsPersist = 256;  // ... and of a combine item of the one-launch kernel
constexpr int kCombPartsPersist = 3;   // 3 x 256 threads = the one-launch work group
constexpr int kSpinLimit = 1 << 20;    // polls (each a device round trip, 1-2 us) before giving up

template <int D, int PARTS, int ROWS, bool PERSIST, typename Plan>
__device__ __forceinline__ void combine_item(const AttnArgs& a, const Plan& p, const int item, float* st) {
  constexpr int SLICES = 4 * D / ROWS;  // 16-byte rows per tile block / rows per item
  static_assert(SLICES >= 1 && 4 * D % ROWS == 0 && ROWS % 64 == 0, "slices of whole waves");
  const int r = find_request(p, item, true);
  const auto rq = p.req[r];
  const int n = rq.nv & 0xffff, L = rq.ctx, T = L + n;
  const int g = a.g;
  const int M = n * g, M32 = (M + 31) & ~31;
  const int nch = (T + p.chunk - 1) / p.chunk;
  int local = item - rq.comb_start;
  const int slice = local % SLICES;
  local /= SLICES;
  const int tiles = M32 / 32;
  const int tile = local % tiles;
  const int hk = local / tiles;
  const int t = (int)threadIdx.x % ROWS;
  const int part = __builtin_amdgcn_readfirstlane((int)threadIdx.x / ROWS);
  const int f = slice * ROWS + t;  // row of the block
  const int lane = f & 63, lc = lane & 31, lh = lane >> 5, q = f >> 6;
  const size_t base = (size_t)rq.part_start + (size_t)hk * nch * M32 + (size_t)tile * 32;

  if constexpr (PERSIST) {
    const int ncg = (M + 255) / 256;
    const int tpg = (tiles + ncg - 1) / ncg;  // tiles per column group, as the main items deal them
    const int cg = tile / tpg;
    const int nct = min(tpg, tiles - cg * tpg);
    int32_t* done = a.sync + kSyncHeader + rq.comb_start + hk * ncg + cg;
    if (threadIdx.x == 0) {
      const int target = nch * nct;
      for (int spin = 0; __hip_atomic_load(done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target; ++spin) {
        // give up after the bound, or (checked every 256 polls) once any wait of this call has
        if (spin >= kSpinLimit ||
            ((spin & 255) == 255 && __hip_atomic_load(a.sync + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
          __hip_atomic_store(a.sync + 2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(8);
      }
      int32_t* started = done + kMaxSyncComb;
      if (__hip_atomic_fetch_add(started, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nct * SLICES - 1) {
        __hip_atomic_store(done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(started, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    lds_barrier();
    asm volatile("" ::: "memory");  // the partial loads stay after the wait
  }

  float m = kNegInf, l = 0.f;
  float o[8];
  for (int e = 0; e < 8; ++e) o[e] = 0.f;
  auto absorb = [&](float mc, float lw, const float (&oc)[8]) {
    const float m_new = fmaxf(m, mc);
    const float a0 = __builtin_amdgcn_exp2f((m - m_new) * a.scale_log2);
    const float a1 = __builtin_amdgcn_exp2f((mc - m_new) * a.scale_log2) * lw;
    l = l * a0 + a1;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = o[e] * a0 + oc[e] * a1;
    m = m_new;
  };
  for (int c0 = part; c0 < nch; c0 += 8 * PARTS) {
    float2 ml[8];
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      ml[u] = make_float2(kNegInf, 0.f);
      v[u] = u32x4{0u, 0u, 0u, 0u};
      const int c = c0 + u * PARTS;
      if (c < nch) {
        const size_t t0 = base + (size_t)c * M32;
        if constexpr (PERSIST) {
          ml[u] = load8_coherent(a.part_ml + 2 * (t0 + lc));
          v[u] = load16_coherent(a.part_o + t0 * D + (size_t)f * 8);
        } else {
          ml[u] = *(const float2*)(a.part_ml + 2 * (t0 + lc));
          v[u] = *(const u32x4*)(a.part_o + t0 * D + (size_t)f * 8);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (ml[u].x == kNegInf) continue;  // no key of that chunk is visible to this column
      float oc[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        oc[2 * e] = __uint_as_float(v[u][e] << 16);
        oc[2 * e + 1] = __uint_as_float(v[u][e] & 0xffff0000u);
      }
      // the chunk's normalised output weighs in with its sum: unnormalised o_c = l_c * oc
      absorb(ml[u].x, ml[u].y, oc);
    }
  }
  // Parts 1.. hand (m, l, normalised o) to part 0.
  if (PARTS > 1 && part > 0) {
    float* s = st + ((part - 1) * 10) * ROWS + t;
    s[0] = m;
    s[ROWS] = l;
    const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s[(2 + e) * ROWS] = o[e] * inv;
  }
  if (PARTS > 1) {
    lds_barrier();
    if (part > 0) return;
  }
#pragma unroll
  for (int j = 0; j < PARTS - 1; ++j) {
    const float* s = st + (j * 10) * ROWS + t;
    const float mj = s[0];
    if (mj == kNegInf) continue;
    float oc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) oc[e] = s[(2 + e) * ROWS];
    absorb(mj, s[ROWS], oc);
  }
  const int gc = tile * 32 + lc;
  if (gc >= M) return;
  const int tok = gc / g;
  const int hh = gc - tok * g;
  const size_t orow = (size_t)(rq.q_start + tok) * a.hq + hk * g + hh;
  const float inv = 1.f / l;
  const int d0 = 32 * (q >> 1) + 16 * (q & 1) + 4 * lh;  // dims d0 .. d0 + 3 and d0 + 8 .. d0 + 11
  u32x2 w0, w1;
  w0[0] = pack_bf16x2(o[0] * inv, o[1] * inv);
  w0[1] = pack_bf16x2(o[2] * inv, o[3] * inv);
  w1[0] = pack_bf16x2(o[4] * inv, o[5] * inv);
  w1[1] = pack_bf16x2(o[6] * inv, o[7] * inv);
  *(u32x2*)(a.out + orow * D + d0) = w0;
  *(u32x2*)(a.out + orow * D + d0 + 8) = w1;
  if (a.lse != nullptr && f < 32) a.lse[orow] = m * a.sm_scale + __logf(l);
}

// Main kernel of the two-launch mode: one work item per work group, in
// dispatch order.  One request: its heads' chunk ranges go to one XCD each
// (shared q and page list in that XCD's L2).  Several: dispatch order, so the
// costliest requests, which come first, spread over all XCDs.
template <int D, typename Plan>
__global__ __launch_bounds__(kThreads) void attn_fwd_kernel(AttnArgs a, Plan p) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[(kKBufs + kVBufs) * kSuper * D];
  const int item = p.num_req == 1 ? xcd_item(p.grid_items) : (int)blockIdx.x;
  if (item >= p.total_items) return;
  attn_item<D, Plan, false>(a, p, item, lds);
}

template <int D, int PARTS, typename Plan>
__global__ __launch_bounds__(kCombRows * PARTS) void attn_combine_kernel(AttnArgs a, Plan p) {
  __shared__ float st[(PARTS > 1 ? PARTS - 1 : 1) * 10 * kCombRows];
  const int item = xcd_item(p.grid_comb);
  if (item >= p.total_comb) return;
  combine_item<D, PARTS, kCombRows, false>(a, p, item, st);
}

// One-launch work-queue kernel (launches with split requests).  The queue
// is every main item (costliest request first), then every combine item.
// Every work group takes every item, its first included, from an atomic
// queue head, so an item is only ever held by a work group that is running,
// and every combine item is taken after every main item: the chunks a
// combine item waits for are all held by running work groups, and a work
// group holding a main item as its next one is busy with a main item, which
// waits for nothing.  A work group asks for its next item at the start of
// the current one, so the queue's latency is hidden.  The combine items of a
// request run in the same launch, as soon as its chunks are done, on work
// groups that would otherwise sit idle or exit: no second launch, and no
// kernel boundary between a split request's chunks and their merge.  The
// last work group to leave returns the queue head and the exit count to
// zero for the next call, and moves a raised give-up flag (sync word 2) to
// the report word (sync word 3), where rg_draft_verify_attention_check finds
// it: the flag does not carry over into the next call.
template <int D, typename Plan>
__global__ __launch_bounds__(kThreads) void attn_persist_kernel(AttnArgs a, Plan p) {
  constexpr int WORDS = (kKBufs + kVBufs) * kSuper * D / 2;  // 32-bit words of LDS (all of it)
  __shared__ __attribute__((aligned(16))) uint16_t lds[(kKBufs + kVBufs) * kSuper * D];
  // The next item's index passes through the last word of the second V
  // buffer: no key-group merge area or combine exchange reaches it, and an
  // item writes that buffer only after its first barrier (buffer 1 goes in
  // before the second one).
  int* const s_next = reinterpret_cast<int*>(lds) + WORDS - 1;
  static_assert(kCombRowsPersist * kCombPartsPersist == kThreads, "combine items use the whole work group");
  static_assert((kCombPartsPersist - 1) * 10 * kCombRowsPersist < WORDS - 1, "combine exchange below the slot");
  static_assert((kWaves - 1) * (64 * 16 * (D / 32) + 128) < WORDS - 1, "key-group merge area below the slot");
  const int total = p.total_items + p.total_comb;
  if (threadIdx.x == 0) *s_next = __hip_atomic_fetch_add(a.sync, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  lds_barrier();
  int item = *s_next;
  while ((unsigned)item < (unsigned)total) {  // (also stops on a queue head that was not zero)
    int nxt = total;
    if (threadIdx.x == 0) nxt = __hip_atomic_fetch_add(a.sync, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (item < p.total_items)
      attn_item<D, Plan, true>(a, p, item, lds);
    else
      combine_item<D, kCombPartsPersist, kCombRowsPersist, true>(a, p, item - p.total_items,
                                                                reinterpret_cast<float*>(lds));
    lds_barrier();  // every wave is done with LDS
    if (threadIdx.x == 0) *s_next = nxt;
    lds_barrier();
    item = *s_next;
  }
  if (threadIdx.x == 0 &&
      __hip_atomic_fetch_add(a.sync + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (int)gridDim.x - 1) {
    __hip_atomic_store(a.sync, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.sync + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int gave_up = __hip_atomic_load(a.sync + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (gave_up != 0) {
      __hip_atomic_store(a.sync + 3, gave_up, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.sync + 2, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int D, typename Plan>
hipError_t launch_impl(const AttnArgs& args, const Plan& plan, hipStream_t stream) {
  if (plan.persist_grid > 0) {
    hipLaunchKernelGGL((attn_persist_kernel<D, Plan>), dim3(plan.persist_grid), dim3(kThreads), 0, stream, args,
                       plan);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((attn_fwd_kernel<D, Plan>), dim3(plan.grid_items), dim3(kThreads), 0, stream, args, plan);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (plan.total_comb > 0) {
    if (plan.max_chunks > 8 && plan.grid_comb <= 1024)  // long rows, and few enough items to be latency-bound
      hipLaunchKernelGGL((attn_combine_kernel<D, 4, Plan>), dim3(plan.grid_comb), dim3(kCombRows * 4), 0, stream, args, plan);
    else
      hipLaunchKernelGGL((attn_combine_kernel<D, 1, Plan>), dim3(plan.grid_comb), dim3(kCombRows), 0, stream, args, plan);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& args, const AttnPlan& plan, int head_dim,
                            hipStream_t stream) {
  if (head_dim == 128) return launch_impl<128>(args, plan, stream);
  return launch_impl<64>(args, plan, stream);
}

hipError_t launch_attention(const AttnArgs& args, const AttnPlanBr& plan, int head_dim,
                            hipStream_t stream) {
  if (head_dim == 128) return launch_impl<128>(args, plan, stream);
  return launch_impl<64>(args, plan, stream);
}

}  // namespace rg

// gfx950 kernels for exact top-k sparsification with error feedback and the
// sparse aggregate + multi-tensor SGD update.
//
// Sparsify (Sec. 3.1 TopK operator, read as exactly k elements with ties to
// the lower position; Alg. 1 output: ascending indices and the values of x):
//   stream   x = g + r stored into r; 11-bit histogram of the magnitude key;
//            one 16-bit max-key summary per 32-element line
//   pick 1   bin of the k-th largest key (one workgroup per group)
//   refine 2 10-bit histogram of the next key bits, only over the lines whose
//            summary can hold a key of the chosen bin
//   pick 2, refine 3, pick 3   the same for the last 10 bits: exact threshold
//            key T and the tie quota `need` (elements equal to T to keep)
//   count    per tile: #{key > T}, #{key == T}
//   scan     exclusive prefix of those counts within each group
//   emit     ordered compaction of the selected (idx, val); r[idx] = +0
// Every step after the stream touches only lines whose summary reaches the
// current key class, so for rho << 1 the data is streamed from HBM once.
//
// Update (Alg. 2 accumulation of the gathered lists; Eq. (1) with optional
// weight decay and momentum):
//   seg      per worker, the first list entry of every update tile (the lists
//            are ascending, so tile boundaries are where idx >> shift grows)
//   update   per tile: LDS accumulation of all workers' entries of the tile,
//            then one pass applying the SGD step to that parameter range
#include <hip/hip_runtime.h>

#include "tkef.h"
#include "tkef_internal.h"

// The update's arithmetic is specified as separate binary32 operations.
#pragma clang fp contract(off)

namespace tkef {

namespace {

__device__ __forceinline__ uint32_t mag_key(float x) {
  return __float_as_uint(x) & 0x7FFFFFFFu;
}

constexpr uint32_t kNanKeyMin = 0x7F800001u;  // keys above +inf's are NaNs

// Exclusive scan of one uint32 per thread across a kBlock-thread workgroup.
// `buf` holds kBlock words of LDS. Returns the exclusive prefix; *total gets
// the sum of all values.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* buf,
                                                    uint32_t* total) {
  const int tid = threadIdx.x;
  buf[tid] = v;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    uint32_t add = (tid >= off) ? buf[tid - off] : 0u;
    __syncthreads();
    buf[tid] += add;
    __syncthreads();
  }
  uint32_t incl = buf[tid];
  *total = buf[kBlock - 1];
  __syncthreads();
  return incl - v;
}

// Loads the elements [e0, e0 + n) of one line (n <= kLine) of x into v[].
__device__ __forceinline__ void load_line(const float* __restrict__ x, int e0, int n,
                                          float (&v)[kLine]) {
  const float* p = x + e0;
  if (n == kLine && (reinterpret_cast<uintptr_t>(p) & 15u) == 0) {
    const float4* p4 = reinterpret_cast<const float4*>(p);
#pragma unroll
    for (int q = 0; q < kLine / 4; ++q) {
      float4 f = p4[q];
      v[4 * q + 0] = f.x;
      v[4 * q + 1] = f.y;
      v[4 * q + 2] = f.z;
      v[4 * q + 3] = f.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < kLine; ++q) v[q] = (q < n) ? p[q] : 0.0f;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
__global__ void k_fill_u32(uint32_t* __restrict__ p, uint32_t v, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += step) p[i] = v;
}

// ---------------------------------------------------------------------------
// stream: x = g + r (stored into r), level-1 histogram, line summaries.
//
// Persistent grid (a few workgroups per CU) walking the tiles in quarters of
// kQuarter elements, so that at any moment the whole GPU streams through one
// compact window of memory. g and r are read with non-temporal loads (each is
// read exactly once); x is stored normally so that the few lines re-read by
// the later steps are likely still cached. Each workgroup keeps an LDS
// histogram and adds it to one of `nslots` copies of its group's global
// histogram when the group changes and at the end; the copies spread the
// atomics of many workgroups over many addresses.
constexpr int kQuarter = 2048;
constexpr int kQuarterLines = kQuarter / kLine;

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 load_nt4(const float4* p) {
  const v4f t = __builtin_nontemporal_load(reinterpret_cast<const v4f*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ void store_nt4(float4* p, float4 v) {
  const v4f t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<v4f*>(p));
}

__device__ __forceinline__ uint32_t add_quad(float4 a, float4 b, float4& x, uint32_t* h) {
  x.x = a.x + b.x;
  x.y = a.y + b.y;
  x.z = a.z + b.z;
  x.w = a.w + b.w;
  const uint32_t k0 = mag_key(x.x), k1 = mag_key(x.y), k2 = mag_key(x.z), k3 = mag_key(x.w);
  atomicAdd(&h[k0 >> kH1Shift], 1u);
  atomicAdd(&h[k1 >> kH1Shift], 1u);
  atomicAdd(&h[k2 >> kH1Shift], 1u);
  atomicAdd(&h[k3 >> kH1Shift], 1u);
  return max(max(k0, k1), max(k2, k3));
}

// Adds the LDS histogram into `dst` and clears it. Called by the whole
// workgroup.
__device__ __forceinline__ void flush_hist(uint32_t* h, uint32_t* __restrict__ dst) {
  __syncthreads();
  for (int i = threadIdx.x; i < kH1Bins; i += kBlock) {
    const uint32_t c = h[i];
    if (c) {
      atomicAdd(&dst[i], c);
      h[i] = 0u;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void k_stream(const TileDesc* __restrict__ tiles,
                                                   int32_t ntiles, uint32_t* __restrict__ hist1,
                                                   int nslots, uint16_t* __restrict__ summ,
                                                   uint32_t* __restrict__ status) {
  __shared__ uint32_t h[kH1Bins];
  __shared__ uint32_t lmax[kQuarterLines];
  __shared__ uint32_t nanflag;
  const int tid = threadIdx.x;
  for (int i = tid; i < kH1Bins; i += kBlock) h[i] = 0u;
  if (tid == 0) nanflag = 0u;
  __syncthreads();
  const int slot = blockIdx.x % nslots;
  const int nunits = ntiles * (kTile / kQuarter);
  int cur = -1;
  uint32_t tmax = 0u;  // largest key this thread saw (NaN check)
  for (int unit = blockIdx.x; unit < nunits; unit += gridDim.x) {
    const TileDesc t = tiles[unit / (kTile / kQuarter)];
    const int s0 = (unit % (kTile / kQuarter)) * kQuarter;
    if (s0 >= t.len) continue;
    const int len = min(kQuarter, t.len - s0);
    if (t.group != cur) {
      if (cur >= 0) flush_hist(h, hist1 + ((size_t)cur * nslots + slot) * kH1Bins);
      cur = t.group;
    }
    const float* __restrict__ g = t.g + s0;
    float* __restrict__ r = t.r + s0;
    uint16_t* __restrict__ sq = summ + (size_t)(unit / (kTile / kQuarter)) * kLinesPerTile +
                                s0 / kLine;
    const bool full = len == kQuarter &&
        ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(r)) & 15u) == 0;
    if (full) {
      // 512 float4 per quarter: two per thread; a line is 8 consecutive lanes
      const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
      float4* __restrict__ r4 = reinterpret_cast<float4*>(r);
      const float4 a0 = load_nt4(g4 + tid), a1 = load_nt4(g4 + kBlock + tid);
      const float4 b0 = load_nt4(r4 + tid), b1 = load_nt4(r4 + kBlock + tid);
      float4 x0, x1;
      uint32_t m0 = add_quad(a0, b0, x0, h);
      uint32_t m1 = add_quad(a1, b1, x1, h);
      store_nt4(r4 + tid, x0);
      store_nt4(r4 + kBlock + tid, x1);
      tmax = max(tmax, max(m0, m1));
      m0 = max(m0, (uint32_t)__shfl_xor((int)m0, 1));
      m1 = max(m1, (uint32_t)__shfl_xor((int)m1, 1));
      m0 = max(m0, (uint32_t)__shfl_xor((int)m0, 2));
      m1 = max(m1, (uint32_t)__shfl_xor((int)m1, 2));
      m0 = max(m0, (uint32_t)__shfl_xor((int)m0, 4));
      m1 = max(m1, (uint32_t)__shfl_xor((int)m1, 4));
      if ((tid & 7) == 0) {
        sq[tid >> 3] = (uint16_t)(m0 >> 16);
        sq[(kBlock + tid) >> 3] = (uint16_t)(m1 >> 16);
      }
    } else {
      // partial or misaligned quarter: element by element, every load issued
      // before the first use so the quarter costs one memory latency
      constexpr int kPer = kQuarter / kBlock;
      if (tid < kQuarterLines) lmax[tid] = 0u;
      __syncthreads();
      float gv[kPer], rv[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        gv[q] = (e < len) ? g[e] : 0.0f;
        rv[q] = (e < len) ? r[e] : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        if (e < len) {
          const float x = gv[q] + rv[q];
          r[e] = x;
          const uint32_t k = mag_key(x);
          atomicAdd(&h[k >> kH1Shift], 1u);
          atomicMax(&lmax[e / kLine], k);
          tmax = max(tmax, k);
        }
      }
      __syncthreads();
      const int nlines = (len + kLine - 1) / kLine;
      if (tid < nlines) sq[tid] = (uint16_t)(lmax[tid] >> 16);
      __syncthreads();
    }
  }
  if (cur >= 0) flush_hist(h, hist1 + ((size_t)cur * nslots + slot) * kH1Bins);
  if (tmax >= kNanKeyMin) atomicOr(&nanflag, 1u);
  __syncthreads();
  if (tid == 0 && nanflag && status) atomicOr(status, TKEF_STATUS_NAN);
}

// ---------------------------------------------------------------------------
// pick: one workgroup per group. Walking the histogram from its highest bin,
// find the bin where the running count first reaches `need`. Each thread owns
// PER consecutive bins, summed over the histogram's `nslots` copies with
// 16-byte loads that are all in flight together.
template <int PER>
__global__ __launch_bounds__(kBlock) void k_pick(int level, const GroupDesc* __restrict__ groups,
                                                 GroupState* __restrict__ st,
                                                 const uint32_t* __restrict__ hist, int nslots) {
  constexpr int nbins = PER * kBlock;
  __shared__ uint32_t part[kBlock];
  __shared__ uint32_t res[3];
  const int g = blockIdx.x, tid = threadIdx.x;
  const GroupState s = st[g];
  const uint32_t need = (level == 1) ? groups[g].k : s.need;
  if (need == 0u) {  // nothing (left) to select in this group
    if (tid == 0) {
      GroupState z;
      z.need = 0u;
      z.prefix = 0xFFFFFFFFu;
      z.T = 0xFFFFFFFFu;
      z.n_eq = 0u;
      st[g] = z;
    }
    return;
  }
  if (tid == 0) {
    res[0] = 0u;
    res[1] = 0u;
    res[2] = 0u;
  }
  // this thread's bins: lo .. lo + PER - 1, threads ordered from the top
  const int lo = nbins - PER * (tid + 1);
  const uint32_t* __restrict__ hg = hist + (size_t)g * nslots * nbins + lo;
  uint32_t c[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) c[j] = 0u;
#pragma unroll 16
  for (int sl = 0; sl < nslots; ++sl) {
    const uint4* p4 = reinterpret_cast<const uint4*>(hg + (size_t)sl * nbins);
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
      const uint4 v = p4[q];
      c[4 * q + 0] += v.x;
      c[4 * q + 1] += v.y;
      c[4 * q + 2] += v.z;
      c[4 * q + 3] += v.w;
    }
  }
  uint32_t sum = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) sum += c[j];
  uint32_t total;
  const uint32_t excl = block_excl_scan(sum, part, &total);
  if (excl < need && need <= excl + sum) {
    uint32_t acc = excl;
#pragma unroll
    for (int j = PER - 1; j >= 0; --j) {  // highest bin first
      if (acc + c[j] >= need) {
        res[0] = (uint32_t)(lo + j);
        res[1] = acc;
        res[2] = c[j];
        break;
      }
      acc += c[j];
    }
  }
  __syncthreads();
  if (tid == 0) {
    const uint32_t bin = res[0], above = res[1], cnt = res[2];
    GroupState ns = s;
    if (level == 1) {
      ns.prefix = bin;
    } else if (level == 2) {
      ns.prefix = (s.prefix << 10) | bin;
    } else {
      ns.T = (s.prefix << 10) | bin;
      ns.n_eq = cnt;
    }
    ns.need = (above < need) ? need - above : 0u;
    st[g] = ns;
  }
}

// ---------------------------------------------------------------------------
// Selection kernels after the level-1 pick (gather, hist3, emit).
//
// They run as at most kSMaxGroups workgroups of kSBlock threads. gather splits
// the summary lines into contiguous ranges, one per workgroup (`lpt` lines per
// thread, in order); hist3 and emit split the compacted candidate list the
// same way (or the lines again, after a candidate overflow). A candidate is
// encoded as (tile << 13) | position-in-tile.
//
// Ordered output needs each workgroup's exclusive prefix of per-workgroup
// counts. Each workgroup publishes its count in a flag word (bit 63 = valid)
// and then reads the words of all lower-numbered workgroups. It waits only on
// workgroups dispatched before it, which publish without waiting on anything,
// so the wait always ends; it is still bounded (kSpinLimit polls per word),
// after which TKEF_STATUS_TIMEOUT is recorded and the workgroup goes on. Flag
// words are cleared before every execution.
constexpr int kSBlock = 1024;
constexpr int kSWaves = kSBlock / 64;
constexpr int kSMaxGroups = 4096;
constexpr int kSMaxLpt = 16;     // lines per thread at most
constexpr int kCandShift = 13;   // log2(kTile)
static_assert((1 << kCandShift) == kTile, "candidate encoding");
constexpr uint64_t kFlagValid = 1ull << 63, kFlagVal = (1ull << 63) - 1;
constexpr uint32_t kSpinLimit = 1u << 22;

__device__ __forceinline__ uint64_t flag_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void flag_store(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, off);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), off);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

// Exclusive scan over a kSBlock-thread workgroup (wave scans + a scan of the
// wave totals). wsum: kSWaves words of LDS. Ends with a barrier.
__device__ __forceinline__ uint32_t sblock_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wid] = x;
  __syncthreads();
  if (wid == 0) {
    uint32_t ws = (lane < kSWaves) ? wsum[lane] : 0u;
#pragma unroll
    for (int off = 1; off < kSWaves; off <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)ws, off);
      if (lane >= off) ws += y;
    }
    if (lane < kSWaves) wsum[lane] = ws;
  }
  __syncthreads();
  const uint32_t before = wid ? wsum[wid - 1] : 0u;
  *total = wsum[kSWaves - 1];
  __syncthreads();
  return before + x - v;
}

// Sum of one u64 per thread over the workgroup. red: kSWaves words of LDS.
__device__ __forceinline__ uint64_t sblock_sum_u64(uint64_t v, uint64_t* red) {
  const int tid = threadIdx.x;
  v = wave_sum_u64(v);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  uint64_t t = 0;
#pragma unroll
  for (int i = 0; i < kSWaves; ++i) t += red[i];
  __syncthreads();
  return t;
}

// Publishes this workgroup's count and returns the sum of the counts of the
// workgroups numbered below it.
__device__ uint64_t group_prefix(uint64_t* __restrict__ flags, uint64_t mine, uint64_t* red,
                                 uint32_t* __restrict__ status) {
  const int tid = threadIdx.x;
  const int w = blockIdx.x;
  if (tid == 0) flag_store(&flags[w], kFlagValid | mine);
  uint64_t v = 0;
  for (int j = tid; j < w; j += kSBlock) {
    uint64_t f = flag_load(&flags[j]);
    uint32_t spins = 0;
    while (!(f & kFlagValid)) {
      if (++spins > kSpinLimit) {
        if (status) atomicOr(status, TKEF_STATUS_TIMEOUT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      f = flag_load(&flags[j]);
    }
    v += f & kFlagVal;
  }
  return sblock_sum_u64(v, red);
}

// Within one workgroup: the bin of a 1024-bin histogram (highest bin first)
// where the running count reaches `need`. res[] (LDS): bin, count above it,
// count in it.
__device__ __forceinline__ void sblock_pick(const uint32_t* __restrict__ hist, uint32_t need,
                                            uint32_t* wsum, uint32_t* res) {
  static_assert(kH2Bins == kSBlock && kH3Bins == kSBlock, "one bin per thread");
  const int tid = threadIdx.x;
  const int bin = kSBlock - 1 - tid;
  const uint32_t c = hist[bin];
  __syncthreads();  // earlier readers of res[] are done
  if (tid == 0) {
    res[0] = 0u;
    res[1] = 0u;
    res[2] = 0u;
  }
  uint32_t total;
  const uint32_t ex = sblock_scan(c, wsum, &total);
  if (ex < need && need <= ex + c) {
    res[0] = (uint32_t)bin;
    res[1] = ex;
    res[2] = c;
  }
  __syncthreads();
}

// Within one workgroup: level-1 pick over a 2048-bin histogram held in
// `nslots` copies (two bins per thread). Returns via res[]: bin, count above
// it, count in it. Ends with a barrier.
__device__ __forceinline__ void sblock_pick1(const uint32_t* __restrict__ hist1, int nslots,
                                             uint32_t need, uint32_t* wsum, uint32_t* res) {
  static_assert(kH1Bins == 2 * kSBlock, "two bins per thread");
  const int tid = threadIdx.x;
  const int lo = kH1Bins - 2 * (tid + 1);  // this thread's bins: lo, lo + 1 (from the top)
  uint32_t c0 = 0u, c1 = 0u;
#pragma unroll 16
  for (int sl = 0; sl < nslots; ++sl) {
    const uint2 v = *reinterpret_cast<const uint2*>(hist1 + (size_t)sl * kH1Bins + lo);
    c0 += v.x;
    c1 += v.y;
  }
  __syncthreads();  // earlier readers of res[] are done
  if (tid == 0) {
    res[0] = 0u;
    res[1] = 0u;
    res[2] = 0u;
  }
  uint32_t total;
  const uint32_t ex = sblock_scan(c0 + c1, wsum, &total);
  if (ex < need && need <= ex + c0 + c1) {
    if (ex + c1 >= need) {  // higher bin first
      res[0] = (uint32_t)(lo + 1);
      res[1] = ex;
      res[2] = c1;
    } else {
      res[0] = (uint32_t)lo;
      res[1] = ex + c1;
      res[2] = c0;
    }
  }
  __syncthreads();
}

// The thread's `lpt` consecutive summary lines starting at line0, seen
// through the (at most two) tiles they lie in. Summaries and descriptors are
// fetched together up front; flagged() gives the lines whose summary reaches
// thr(group).
struct LineSpan {
  int64_t line0, last;
  int tile0, tile1;
  TileDesc tA, tB;
  uint16_t sv[kSMaxLpt];

  __device__ __forceinline__ void load(const TileDesc* __restrict__ tiles,
                                       const uint16_t* __restrict__ summ, int64_t nlines,
                                       int64_t l0, int lpt) {
    line0 = l0;
    const bool has = l0 < nlines;
    last = has ? min(l0 + lpt, nlines) - 1 : l0 - 1;
    tile0 = has ? (int)(l0 / kLinesPerTile) : 0;
    tile1 = has ? (int)(last / kLinesPerTile) : 0;
#pragma unroll
    for (int q = 0; q < kSMaxLpt; ++q) sv[q] = (l0 + q <= last) ? summ[l0 + q] : (uint16_t)0;
    tA = tiles[tile0];
    tB = tiles[tile1];
  }
  __device__ __forceinline__ bool in_a(int q) const {
    return (int)((line0 + q) / kLinesPerTile) == tile0;
  }
  __device__ __forceinline__ const TileDesc& desc(int q) const { return in_a(q) ? tA : tB; }
  __device__ __forceinline__ int tile(int q) const { return in_a(q) ? tile0 : tile1; }
  __device__ __forceinline__ int e0(int q) const {
    return (int)((line0 + q) % kLinesPerTile) * kLine;
  }
  template <typename Thr>
  __device__ __forceinline__ uint32_t flagged(Thr thr) const {
    const uint32_t ta = thr(tA.group) >> 16, tb = thr(tB.group) >> 16;
    uint32_t m = 0u;
#pragma unroll
    for (int q = 0; q < kSMaxLpt; ++q) {
      const bool a = in_a(q);
      if (line0 + q <= last && e0(q) < (a ? tA.len : tB.len) && (uint32_t)sv[q] >= (a ? ta : tb))
        m |= 1u << q;
    }
    return m;
  }
};

// For every element of the flagged lines in `mask`, in position order, for
// which hit(group, key) holds: f(tile, TileDesc, e, x, key). The hit test runs
// over all 32 elements of a line at once; the (few) hits are then visited one
// by one, re-reading the element from the line just loaded.
template <typename Hit, typename F>
__device__ __forceinline__ void walk_mask(const LineSpan& ls, uint32_t mask, Hit hit, F f) {
#pragma unroll 1
  while (mask) {
    const int q = __ffs(mask) - 1;
    mask &= mask - 1u;
    const TileDesc& t = ls.desc(q);
    const int e0 = ls.e0(q), n = min(kLine, t.len - e0);
    float v[kLine];
    load_line(t.r, e0, n, v);
    uint32_t hm = 0u;
#pragma unroll
    for (int j = 0; j < kLine; ++j)
      hm |= (j < n && hit(t.group, mag_key(v[j]))) ? (1u << j) : 0u;
    const int tile = ls.tile(q);
#pragma unroll 1
    while (hm) {
      const int j = __ffs(hm) - 1;
      hm &= hm - 1u;
      const float x = t.r[e0 + j];
      f(tile, t, e0 + j, x, mag_key(x));
    }
  }
}

// Calls f(tile, TileDesc, e, x, key) for candidates [cb, ce), in order.
template <typename F>
__device__ __forceinline__ void walk_cands(const TileDesc* __restrict__ tiles, int32_t ntiles,
                                           const int32_t* __restrict__ cand, uint32_t cb,
                                           uint32_t ce, F f) {
#pragma unroll 1
  for (uint32_t j = cb; j < ce; ++j) {
    const uint32_t c = (uint32_t)cand[j];
    const int tile = (int)(c >> kCandShift);
    const int e = (int)(c & (kTile - 1));
    if (tile >= ntiles) continue;  // never produced; keeps accesses in bounds
    const TileDesc t = tiles[tile];
    if (e >= t.len) continue;
    const float x = t.r[e];
    f(tile, t, e, x, mag_key(x));
  }
}

// ---------------------------------------------------------------------------
// gather: after the level-1 pick. Over the lines whose summary can hold a key
// of at least the chosen bin B1: (a) histogram of key bits 19..10 of the
// elements in bin B1 (level 2); (b) ordered compaction of all elements with
// key >= B1 << 20 into `cand`. meta[0] = overflow (the candidates did not fit
// in `cap`; later steps then read lines), meta[1] = candidate count.
constexpr int kStage = 8;  // candidates / items a thread stages in LDS

__global__ __launch_bounds__(kSBlock) void k_gather(const TileDesc* __restrict__ tiles,
                                                    const GroupDesc* __restrict__ groups,
                                                    GroupState* __restrict__ st,
                                                    const uint32_t* __restrict__ hist1, int nslots,
                                                    int single, const uint16_t* __restrict__ summ,
                                                    int64_t nlines, int lpt,
                                                    uint32_t* __restrict__ hist2,
                                                    uint64_t* __restrict__ flags,
                                                    int32_t* __restrict__ cand, uint32_t cap,
                                                    uint32_t* __restrict__ meta,
                                                    uint32_t* __restrict__ status) {
  __shared__ uint32_t h[kH2Bins];
  __shared__ uint32_t wsum[kSWaves];
  __shared__ uint64_t red[kSWaves];
  __shared__ uint32_t res[3];
  __shared__ int32_t stage[kStage * kSBlock];  // [slot][thread]
  __shared__ uint32_t any;
  const int tid = threadIdx.x;
  h[tid] = 0u;
  if (tid == 0) any = 0u;

  // 1. summaries and tiles of this thread's lines (independent of the pick)
  LineSpan ls;
  ls.load(tiles, summ, nlines, ((int64_t)blockIdx.x * kSBlock + tid) * lpt, lpt);

  // 2. level-1 pick. One selection group: every workgroup makes it itself
  //    from the slotted histogram and workgroup 0 records it for the later
  //    kernels. Several groups: the pick kernel has done it.
  GroupState s0;
  if (single) {
    const uint32_t k = groups[0].k;
    sblock_pick1(hist1, nslots, k, wsum, res);
    s0.prefix = (k == 0u) ? 0xFFFFFFFFu : res[0];
    s0.need = (k == 0u || res[1] >= k) ? 0u : k - res[1];
    s0.T = 0xFFFFFFFFu;
    s0.n_eq = 0u;
    if (blockIdx.x == 0 && tid == 0) st[0] = s0;
  } else {
    s0 = st[0];
  }
  // B1 = 0xFFFFFFFF for a group with nothing to select: shifted, it lies
  // above every key, so such a group yields no candidates
  auto b1_of = [&](int g) -> uint32_t { return single ? s0.prefix : st[g].prefix; };
  const uint32_t b1A = b1_of(ls.tA.group), b1B = b1_of(ls.tB.group);
  const uint32_t mask = ls.flagged([&](int g) -> uint32_t {
    return (g == ls.tA.group ? b1A : b1B) << kH1Shift;
  });

  // 3. count the candidates of the flagged lines; stage the first kStage in LDS
  auto is_cand = [&](int g, uint32_t k) -> bool {
    return k >= ((g == ls.tA.group ? b1A : b1B) << kH1Shift);
  };
  uint32_t c = 0u, hit = 0u;
  walk_mask(ls, mask, is_cand, [&](int tile, const TileDesc& t, int e, float, uint32_t k) {
    const uint32_t b1 = (t.group == ls.tA.group) ? b1A : b1B;
    if (c < (uint32_t)kStage)
      stage[c * kSBlock + tid] = (int32_t)(((uint32_t)tile << kCandShift) | (uint32_t)e);
    ++c;
    if ((k >> kH1Shift) == b1) {
      const uint32_t bin = (k >> kH2Shift) & (kH2Bins - 1);
      if (single) atomicAdd(&h[bin], 1u);
      else atomicAdd(&hist2[(size_t)t.group * kH2Bins + bin], 1u);
      hit = 1u;
    }
  });
  if (hit) any = 1u;

  // 4. ordered positions: scan within the workgroup, prefix across workgroups
  uint32_t total;
  const uint32_t ex = sblock_scan(c, wsum, &total);
  const uint64_t pre = group_prefix(flags, total, red, status);
  const bool fits = pre + total <= cap;
  if (tid == 0) {
    if (!fits) atomicOr(&meta[0], 1u);
    if (blockIdx.x == gridDim.x - 1) meta[1] = (uint32_t)min(pre + total, (uint64_t)0xFFFFFFFFu);
  }
  if (fits && c) {
    const uint64_t pos = pre + ex;
    const uint32_t ns = min(c, (uint32_t)kStage);
#pragma unroll 1
    for (uint32_t q = 0; q < ns; ++q) cand[pos + q] = stage[q * kSBlock + tid];
    if (c > (uint32_t)kStage) {  // rare: read the lines again for the rest
      uint32_t i = 0u;
      walk_mask(ls, mask, is_cand, [&](int tile, const TileDesc&, int e, float, uint32_t) {
        if (i >= (uint32_t)kStage)
          cand[pos + i] = (int32_t)(((uint32_t)tile << kCandShift) | (uint32_t)e);
        ++i;
      });
    }
  }
  if (single && any) {  // `any` was written before the scans' barriers
    const uint32_t v = h[tid];
    if (v) atomicAdd(&hist2[tid], v);
  }
}

// Level-2 state of a group: redundant per workgroup for a single group (from
// the level-2 histogram), else written by the pick kernel.
__device__ __forceinline__ void sel_level2(const GroupState& s1, const uint32_t* __restrict__ hist2,
                                           uint32_t* wsum, uint32_t* res, uint32_t* cls21,
                                           uint32_t* need2) {
  sblock_pick(hist2, s1.need, wsum, res);
  *cls21 = (s1.prefix << 10) | res[0];
  *need2 = (res[1] < s1.need) ? s1.need - res[1] : 0u;
}

// ---------------------------------------------------------------------------
// hist3: histogram of the low 10 key bits over the level-2 class
// (key >> 10 == prefix of 21 bits), read from the candidates (or the lines).
__global__ __launch_bounds__(kSBlock) void k_hist3(const TileDesc* __restrict__ tiles,
                                                   int32_t ntiles,
                                                   const GroupState* __restrict__ st,
                                                   int single, const uint16_t* __restrict__ summ,
                                                   int64_t nlines, int lpt,
                                                   const uint32_t* __restrict__ hist2,
                                                   const int32_t* __restrict__ cand,
                                                   const uint32_t* __restrict__ meta,
                                                   uint32_t* __restrict__ hist3) {
  __shared__ uint32_t h[kH3Bins];
  __shared__ uint32_t wsum[kSWaves];
  __shared__ uint32_t res[3];
  __shared__ uint32_t any;
  const int tid = threadIdx.x;
  const uint32_t ov = meta[0], C = meta[1];
  const GroupState s0 = st[0];
  h[tid] = 0u;
  if (tid == 0) any = 0u;
  uint32_t cls_single = 0xFFFFFFFFu, need_single = 0u;
  if (single) {
    sel_level2(s0, hist2, wsum, res, &cls_single, &need_single);
  } else {
    __syncthreads();
  }
  auto cls_of = [&](int g) -> uint32_t {
    if (single) return need_single ? cls_single : 0xFFFFFFFFu;
    const GroupState sg = st[g];
    return sg.need ? sg.prefix : 0xFFFFFFFFu;
  };
  uint32_t hit = 0u;
  auto in_cls = [&](int g, uint32_t k) -> bool { return (k >> kH2Shift) == cls_of(g); };
  auto body = [&](int, const TileDesc& t, int, float, uint32_t k) {
    if (in_cls(t.group, k)) {
      const uint32_t bin = k & (kH3Bins - 1);
      if (single) atomicAdd(&h[bin], 1u);
      else atomicAdd(&hist3[(size_t)t.group * kH3Bins + bin], 1u);
      hit = 1u;
    }
  };
  if (ov) {
    LineSpan ls;
    ls.load(tiles, summ, nlines, ((int64_t)blockIdx.x * kSBlock + tid) * lpt, lpt);
    walk_mask(ls, ls.flagged([&](int g) -> uint32_t { return cls_of(g) << kH2Shift; }), in_cls,
              body);
  } else {
    const uint32_t per_wg = (C + gridDim.x - 1) / gridDim.x;
    const uint32_t wb = min(C, blockIdx.x * per_wg), we = min(C, wb + per_wg);
#pragma unroll 1
    for (uint32_t j = wb + tid; j < we; j += kSBlock) walk_cands(tiles, ntiles, cand, j, j + 1, body);
  }
  if (hit) any = 1u;
  __syncthreads();
  if (single && any) {
    const uint32_t v = h[tid];
    if (v) atomicAdd(&hist3[tid], v);
  }
}

// ---------------------------------------------------------------------------
// groupscan (per-tensor selections only): base[2g] = sum over earlier groups
// of #{key > T}, base[2g + 1] = the same for #{key == T}.
__global__ __launch_bounds__(kSBlock) void k_groupscan(const GroupDesc* __restrict__ groups,
                                                       const GroupState* __restrict__ st,
                                                       int32_t ngroups,
                                                       uint32_t* __restrict__ base) {
  __shared__ uint32_t wsum[kSWaves];
  const int tid = threadIdx.x;
  uint32_t carry_gt = 0u, carry_eq = 0u;
  for (int g0 = 0; g0 < ngroups; g0 += kSBlock) {
    const int g = g0 + tid;
    uint32_t gt = 0u, eq = 0u;
    if (g < ngroups) {
      const GroupState s = st[g];
      const uint32_t k = groups[g].k;
      gt = (k > s.need) ? k - s.need : 0u;
      eq = s.need ? s.n_eq : 0u;
    }
    uint32_t tg, te;
    const uint32_t xg = sblock_scan(gt, wsum, &tg);
    const uint32_t xe = sblock_scan(eq, wsum, &te);
    if (g < ngroups) {
      base[2 * g] = carry_gt + xg;
      base[2 * g + 1] = carry_eq + xe;
    }
    carry_gt += tg;
    carry_eq += te;
  }
}

// ---------------------------------------------------------------------------
// emit: ordered compaction of the selection. An element of group g with
// key > T_g goes to slot (#gt before it in g) + min(#eq before it in g, need_g);
// an element with key == T_g is kept while fewer than need_g equal keys
// precede it in g. Counts before an element are global prefixes (over the
// candidate list, in position order) minus the group's base.
__global__ __launch_bounds__(kSBlock) void k_emit(const TileDesc* __restrict__ tiles,
                                                  int32_t ntiles,
                                                  const GroupDesc* __restrict__ groups,
                                                  const GroupState* __restrict__ st, int single,
                                                  const uint16_t* __restrict__ summ,
                                                  int64_t nlines, int lpt,
                                                  const uint32_t* __restrict__ hist2,
                                                  const uint32_t* __restrict__ hist3,
                                                  const int32_t* __restrict__ cand,
                                                  const uint32_t* __restrict__ meta,
                                                  const uint32_t* __restrict__ base,
                                                  uint64_t* __restrict__ flags,
                                                  int32_t* __restrict__ idx_out,
                                                  float* __restrict__ val_out,
                                                  uint32_t* __restrict__ status,
                                                  uint32_t* __restrict__ clear_next,
                                                  int64_t clear_words) {
  __shared__ uint32_t wsum[kSWaves];
  __shared__ uint64_t red[kSWaves];
  __shared__ uint32_t res[3];
  __shared__ int32_t stage_code[kStage * kSBlock];  // [slot][thread]: (tile << 13) | e
  __shared__ float stage_x[kStage * kSBlock];
  const int tid = threadIdx.x;
  // clear the other copy of the zero-initialised scratch for the next run
#pragma unroll 1
  for (int64_t i = (int64_t)blockIdx.x * kSBlock + tid; i < clear_words;
       i += (int64_t)gridDim.x * kSBlock)
    clear_next[i] = 0u;
  const uint32_t ov = meta[0], C = meta[1];
  const GroupState s0 = st[0];
  const GroupDesc gd0 = groups[0];
  uint32_t T_one = 0xFFFFFFFFu, need_one = 0u;
  if (single) {
    uint32_t cls21, need2;
    sel_level2(s0, hist2, wsum, res, &cls21, &need2);
    sblock_pick(hist3, need2, wsum, res);
    if (s0.need != 0u && need2 != 0u) {
      T_one = (cls21 << 10) | res[0];
      need_one = (res[1] < need2) ? need2 - res[1] : 0u;
    }
  }
  auto T_of = [&](int g) -> uint32_t { return single ? T_one : st[g].T; };
  // this thread's elements: a run of candidates, or (after an overflow) lines
  LineSpan ls;
  uint32_t mask = 0u, cb = 0u, ce = 0u;
  if (ov) {
    ls.load(tiles, summ, nlines, ((int64_t)blockIdx.x * kSBlock + tid) * lpt, lpt);
    mask = ls.flagged(T_of);
  } else {
    const uint32_t per_wg = (C + gridDim.x - 1) / gridDim.x;
    const uint32_t wb = min(C, blockIdx.x * per_wg), we = min(C, wb + per_wg);
    const uint32_t per = (we - wb + kSBlock - 1) / kSBlock;
    cb = min(we, wb + tid * per);
    ce = min(we, cb + per);
  }
  // pass 1: counts of (key > T) and (key == T), in position order; the first
  // kStage elements with key >= T are staged in LDS for pass 2
  uint32_t gt = 0u, eq = 0u, nst = 0u;
  auto count = [&](int tile, const TileDesc& t, int e, float x, uint32_t k) {
    const uint32_t T = T_of(t.group);
    if (k >= T) {
      if (nst < (uint32_t)kStage) {
        stage_code[nst * kSBlock + tid] = (int32_t)(((uint32_t)tile << kCandShift) | (uint32_t)e);
        stage_x[nst * kSBlock + tid] = x;
      }
      ++nst;
      gt += (k > T) ? 1u : 0u;
      eq += (k == T) ? 1u : 0u;
    }
  };
  auto at_least_T = [&](int g, uint32_t k) -> bool { return k >= T_of(g); };
  if (ov) walk_mask(ls, mask, at_least_T, count);
  else walk_cands(tiles, ntiles, cand, cb, ce, count);
  uint32_t tot_gt, tot_eq;
  const uint32_t xg = sblock_scan(gt, wsum, &tot_gt);
  const uint32_t xe = sblock_scan(eq, wsum, &tot_eq);
  const uint64_t pre = group_prefix(flags, (uint64_t)tot_gt | ((uint64_t)tot_eq << 31), red, status);
  if (nst == 0u) return;
  uint32_t gtr = (uint32_t)(pre & 0x7FFFFFFFu) + xg;
  uint32_t eqr = (uint32_t)((pre >> 31) & 0x7FFFFFFFu) + xe;
  // pass 2: write
  auto write = [&](int, const TileDesc& t, int e, float x, uint32_t k) {
    const int g = t.group;
    const uint32_t T = T_of(g);
    if (k < T) return;
    const GroupDesc gd = single ? gd0 : groups[g];
    const uint32_t need = single ? need_one : st[g].need;
    const uint32_t bg = single ? 0u : base[2 * g], be = single ? 0u : base[2 * g + 1];
    uint32_t pos = 0xFFFFFFFFu;
    if (k > T) {
      pos = (gtr - bg) + min(eqr - be, need);
      ++gtr;
    } else {
      if (eqr - be < need) pos = (gtr - bg) + (eqr - be);
      ++eqr;
    }
    if (pos < gd.k) {
      idx_out[gd.out_base + pos] = t.gstart + e;
      val_out[gd.out_base + pos] = x;
      t.r[e] = 0.0f;
    }
  };
  if (nst <= (uint32_t)kStage) {
#pragma unroll 1
    for (uint32_t q = 0; q < nst; ++q) {
      const uint32_t code = (uint32_t)stage_code[q * kSBlock + tid];
      const int tile = (int)(code >> kCandShift);
      const TileDesc t = tiles[tile];
      const float x = stage_x[q * kSBlock + tid];
      write(tile, t, (int)(code & (kTile - 1)), x, mag_key(x));
    }
  } else if (ov) {
    walk_mask(ls, mask, at_least_T, write);
  } else {
    walk_cands(tiles, ntiles, cand, cb, ce, write);
  }
}

// ---------------------------------------------------------------------------
// seg: seg[u * P + p] = first entry of worker p's list whose index lies in
// update tile u or later; seg[ntiles_u * P + p] = nnz_p. Tile-major, so the
// workgroup of tile u reads two contiguous rows. Also flags unsorted or
// out-of-range lists in the status word.
__global__ void k_seg(const int32_t* __restrict__ idx, int64_t stride,
                      const int32_t* __restrict__ nnz, int32_t P, int32_t d, int32_t ntiles_u,
                      int32_t* __restrict__ seg, uint32_t* __restrict__ status) {
  const int p = blockIdx.y;
  int64_t n = nnz ? (int64_t)nnz[p] : stride;
  n = n < 0 ? 0 : (n > stride ? stride : n);
  const int32_t* __restrict__ L = idx + (int64_t)p * stride;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n == 0) {
    for (int64_t u = j; u <= ntiles_u; u += (int64_t)gridDim.x * blockDim.x)
      seg[u * P + p] = 0;
    return;
  }
  if (j >= n) return;
  auto tile_of = [&](int32_t i) -> int32_t {
    return i < 0 ? 0 : (i >= d ? ntiles_u - 1 : (i >> kUShift));
  };
  const int32_t i = L[j];
  uint32_t bad = (i < 0 || i >= d) ? TKEF_STATUS_INDEX_RANGE : 0u;
  const int32_t t = tile_of(i);
  int32_t tp = -1;
  if (j > 0) {
    const int32_t ip = L[j - 1];
    if (ip > i) bad |= TKEF_STATUS_UNSORTED;
    tp = tile_of(ip);
  }
  for (int32_t u = tp + 1; u <= t; ++u) seg[(int64_t)u * P + p] = (int32_t)j;
  if (j == n - 1)
    for (int32_t u = t + 1; u <= ntiles_u; ++u) seg[(int64_t)u * P + p] = (int32_t)n;
  if (bad && status) atomicOr(status, bad);
}

// ---------------------------------------------------------------------------
// update: one workgroup per update tile.
__device__ __forceinline__ float sgd_step(float G, float w, float& b, bool mom, float lr,
                                          float mu, float wd) {
  const float decay = wd * w;
  const float D = G + decay;
  float U = D;
  if (mom) {
    const float keep = mu * b;
    b = keep + D;
    U = b;
  }
  const float stepv = lr * U;
  return w - stepv;
}

constexpr int kXcds = 8;                      // MI355X: 8 accelerator dies
constexpr int kUVecPerThread = kUTile / 4 / kUBlock;  // float4 per thread per tile

__global__ __launch_bounds__(kUBlock) void k_update(
    const UpdTensor* __restrict__ tens, const int32_t* __restrict__ tile_first, int32_t ntens,
    int32_t d, int32_t ntiles_u, int32_t per_xcd, const int32_t* __restrict__ idx,
    const float* __restrict__ val, int64_t stride, const int32_t* __restrict__ nnz, int32_t P,
    const int32_t* __restrict__ seg, float lr, float mu, float wd, int sparse_mode,
    int has_mom) {
  __shared__ __align__(16) float acc[kUTile];
  __shared__ uint32_t mask[kUTile / 32];
  __shared__ int32_t sbeg[kUBlock];
  __shared__ uint32_t scan[kUBlock];
  const int tid = threadIdx.x;
  // Workgroups go round-robin to the XCDs; give each XCD a contiguous run of
  // tiles so that neighbouring tiles, which share the cache lines at the ends
  // of every worker's list segment, are served by one L2.
  const int u = (int)(blockIdx.x % kXcds) * per_xcd + (int)(blockIdx.x / kXcds);
  if (u >= ntiles_u) return;
  const int32_t base = u << kUShift;
  const int32_t len = min(kUTile, d - base);
  const bool mom = has_mom != 0;

  // Dense fast path: the tile lies inside one tensor and its w (and b) start
  // 16-byte aligned. Its parameters are fetched before the accumulation so
  // their HBM latency overlaps it.
  const int32_t t0 = tile_first[u];
  const UpdTensor tt0 = tens[t0];
  float* __restrict__ w_tile = tt0.w + (base - tt0.goff);
  float* __restrict__ b_tile = mom ? tt0.b + (base - tt0.goff) : nullptr;
  const bool fast = !sparse_mode && len == kUTile && tt0.goff <= base &&
                    (int64_t)base + len <= tt0.goff + tt0.n &&
                    ((reinterpret_cast<uintptr_t>(w_tile) |
                      (mom ? reinterpret_cast<uintptr_t>(b_tile) : 0u)) & 15u) == 0;
  float4 wv[kUVecPerThread], bv[kUVecPerThread];
  if (fast) {
    const float4* w4 = reinterpret_cast<const float4*>(w_tile);
    const float4* b4 = reinterpret_cast<const float4*>(b_tile);
#pragma unroll
    for (int q = 0; q < kUVecPerThread; ++q) {
      wv[q] = load_nt4(w4 + q * kUBlock + tid);
      if (mom) bv[q] = load_nt4(b4 + q * kUBlock + tid);
    }
  }

  for (int i = tid; i < kUTile; i += kUBlock) acc[i] = 0.0f;
  if (sparse_mode)
    for (int i = tid; i < kUTile / 32; i += kUBlock) mask[i] = 0u;
  __syncthreads();

  // 1. accumulate every worker's entries that fall in this tile
  for (int p0 = 0; p0 < P; p0 += kUBlock) {
    const int p = p0 + tid;
    int32_t b = 0, e = 0;
    if (p < P) {
      int64_t np = nnz ? (int64_t)nnz[p] : stride;
      np = np < 0 ? 0 : (np > stride ? stride : np);
      int64_t sb = seg[(int64_t)u * P + p], se = seg[(int64_t)(u + 1) * P + p];
      sb = sb < 0 ? 0 : (sb > np ? np : sb);
      se = se < sb ? sb : (se > np ? np : se);
      b = (int32_t)sb;
      e = (int32_t)se;
    }
    sbeg[tid] = b;
    // inclusive prefix of the segment lengths, for the entry -> worker search
    // (block_excl_scan ends with a barrier, so scan[] can be rewritten here)
    uint32_t total;
    const uint32_t ex = block_excl_scan((uint32_t)(e - b), scan, &total);
    scan[tid] = ex + (uint32_t)(e - b);
    __syncthreads();
    // entries of this batch of workers, kPairUnroll per thread with all
    // their loads in flight before the LDS adds
    constexpr int kPairUnroll = 4;
    for (uint32_t q0 = 0; q0 < total; q0 += kUBlock * kPairUnroll) {
      int32_t li[kPairUnroll];
      float vv[kPairUnroll];
#pragma unroll
      for (int j = 0; j < kPairUnroll; ++j) {
        const uint32_t q = q0 + j * kUBlock + tid;
        li[j] = -1;
        vv[j] = 0.0f;
        if (q < total) {
          int lo = 0, hi = kUBlock - 1;
          while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (scan[mid] > q) hi = mid; else lo = mid + 1;
          }
          const uint32_t before = lo ? scan[lo - 1] : 0u;
          const int64_t gi = (int64_t)(p0 + lo) * stride + sbeg[lo] + (q - before);
          li[j] = idx[gi] - base;
          vv[j] = val[gi];
        }
      }
#pragma unroll
      for (int j = 0; j < kPairUnroll; ++j) {
        if (li[j] >= 0 && li[j] < len) {
          atomicAdd(&acc[li[j]], vv[j]);
          if (sparse_mode) atomicOr(&mask[li[j] >> 5], 1u << (li[j] & 31));
        }
      }
    }
    __syncthreads();
  }

  // 2. apply the SGD step
  if (fast) {
    float4* w4 = reinterpret_cast<float4*>(w_tile);
    float4* b4 = reinterpret_cast<float4*>(b_tile);
    const float4* a4 = reinterpret_cast<const float4*>(acc);
#pragma unroll
    for (int q = 0; q < kUVecPerThread; ++q) {
      const int v = q * kUBlock + tid;
      const float4 G = a4[v];
      float4 w = wv[q], bb = mom ? bv[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      w.x = sgd_step(G.x, w.x, bb.x, mom, lr, mu, wd);
      w.y = sgd_step(G.y, w.y, bb.y, mom, lr, mu, wd);
      w.z = sgd_step(G.z, w.z, bb.z, mom, lr, mu, wd);
      w.w = sgd_step(G.w, w.w, bb.w, mom, lr, mu, wd);
      store_nt4(w4 + v, w);
      if (mom) store_nt4(b4 + v, bb);
    }
    return;
  }
  const int32_t t1 = min(tile_first[u + 1], ntens - 1);
  if (sparse_mode) {
    for (int wi = tid; wi < (len + 31) / 32; wi += kUBlock) {
      uint32_t m = mask[wi];
      while (m) {
        const int bit = __ffs(m) - 1;
        m &= m - 1u;
        const int li = wi * 32 + bit;
        const int64_t gi = (int64_t)base + li;
        int lo = t0, hi = t1;  // last tensor with goff <= gi
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (tens[mid].goff <= gi) lo = mid; else hi = mid - 1;
        }
        float* wp = tens[lo].w + (gi - tens[lo].goff);
        const float stepv = lr * acc[li];
        *wp = *wp - stepv;
      }
    }
    return;
  }
  for (int ti = t0; ti < ntens; ++ti) {
    const UpdTensor tt = tens[ti];
    if (tt.goff >= (int64_t)base + len) break;
    const int64_t a = max((int64_t)base, tt.goff);
    const int64_t z = min((int64_t)base + len, tt.goff + tt.n);
    if (z <= a) continue;
    const int cnt = (int)(z - a);
    const int la = (int)(a - base);
    float* __restrict__ w = tt.w + (a - tt.goff);
    float* __restrict__ bm = mom ? tt.b + (a - tt.goff) : nullptr;
    const bool vec = ((reinterpret_cast<uintptr_t>(w) |
                       (bm ? reinterpret_cast<uintptr_t>(bm) : 0u)) & 15u) == 0;
    int done = 0;
    if (vec) {
      const int nv = cnt >> 2;
      float4* w4 = reinterpret_cast<float4*>(w);
      float4* b4 = reinterpret_cast<float4*>(bm);
      for (int q = tid; q < nv; q += kUBlock) {
        float4 wq = w4[q];
        float4 bq = bm ? b4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
        const int l = la + 4 * q;
        wq.x = sgd_step(acc[l + 0], wq.x, bq.x, mom, lr, mu, wd);
        wq.y = sgd_step(acc[l + 1], wq.y, bq.y, mom, lr, mu, wd);
        wq.z = sgd_step(acc[l + 2], wq.z, bq.z, mom, lr, mu, wd);
        wq.w = sgd_step(acc[l + 3], wq.w, bq.w, mom, lr, mu, wd);
        w4[q] = wq;
        if (mom) b4[q] = bq;
      }
      done = nv << 2;
    }
    for (int q = done + tid; q < cnt; q += kUBlock) {
      float bq = mom ? bm[q] : 0.0f;
      w[q] = sgd_step(acc[la + q], w[q], bq, mom, lr, mu, wd);
      if (mom) bm[q] = bq;
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t launch_stream(const TileDesc* tiles, int32_t ntiles, int32_t grid, uint32_t* hist1,
                         int32_t nslots, uint16_t* summ, uint32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(k_stream, dim3(grid), dim3(kBlock), 0, s, tiles, ntiles, hist1, nslots,
                     summ, status);
  return hipGetLastError();
}

hipError_t launch_pick(int level, const GroupDesc* groups, GroupState* st,
                       const uint32_t* hist, int32_t nslots, int32_t ngroups, hipStream_t s) {
  static_assert(kH1Bins == 8 * kBlock && kH2Bins == 4 * kBlock && kH3Bins == 4 * kBlock,
                "pick: bins per thread");
  if (level == 1)
    hipLaunchKernelGGL(k_pick<8>, dim3(ngroups), dim3(kBlock), 0, s, level, groups, st, hist,
                       nslots);
  else
    hipLaunchKernelGGL(k_pick<4>, dim3(ngroups), dim3(kBlock), 0, s, level, groups, st, hist,
                       nslots);
  return hipGetLastError();
}

hipError_t launch_gather(const TileDesc* tiles, const GroupDesc* groups, GroupState* st,
                         const uint32_t* hist1, int nslots, int single, const uint16_t* summ,
                         int64_t nlines, int lpt, int32_t grid, uint32_t* hist2,
                         uint64_t* flags, int32_t* cand, uint32_t cap, uint32_t* meta,
                         uint32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(k_gather, dim3(grid), dim3(kSBlock), 0, s, tiles, groups, st, hist1, nslots,
                     single, summ, nlines, lpt, hist2, flags, cand, cap, meta, status);
  return hipGetLastError();
}

hipError_t launch_hist3(const TileDesc* tiles, int32_t ntiles, const GroupState* st,
                        int single, const uint16_t* summ, int64_t nlines, int lpt, int32_t grid,
                        const uint32_t* hist2, const int32_t* cand, const uint32_t* meta,
                        uint32_t* hist3, hipStream_t s) {
  hipLaunchKernelGGL(k_hist3, dim3(grid), dim3(kSBlock), 0, s, tiles, ntiles, st, single, summ,
                     nlines, lpt, hist2, cand, meta, hist3);
  return hipGetLastError();
}

hipError_t launch_groupscan(const GroupDesc* groups, const GroupState* st, int32_t ngroups,
                            uint32_t* base, hipStream_t s) {
  hipLaunchKernelGGL(k_groupscan, dim3(1), dim3(kSBlock), 0, s, groups, st, ngroups, base);
  return hipGetLastError();
}

hipError_t launch_emit(const TileDesc* tiles, int32_t ntiles, const GroupDesc* groups,
                       const GroupState* st, int single, const uint16_t* summ, int64_t nlines,
                       int lpt, int32_t grid, const uint32_t* hist2, const uint32_t* hist3,
                       const int32_t* cand, const uint32_t* meta, const uint32_t* base,
                       uint64_t* flags, int32_t* idx_out, float* val_out, uint32_t* status,
                       uint32_t* clear_next, int64_t clear_words, hipStream_t s) {
  hipLaunchKernelGGL(k_emit, dim3(grid), dim3(kSBlock), 0, s, tiles, ntiles, groups, st, single, summ,
                     nlines, lpt, hist2, hist3, cand, meta, base, flags, idx_out, val_out,
                     status, clear_next, clear_words);
  return hipGetLastError();
}

int32_t select_max_groups() { return kSMaxGroups; }
int32_t select_block() { return kSBlock; }
int32_t select_max_lpt() { return kSMaxLpt; }

hipError_t launch_seg(const int32_t* idx, int64_t stride, const int32_t* nnz, int32_t P,
                      int32_t d, int32_t ntiles_u, int32_t* seg, uint32_t* status,
                      hipStream_t s) {
  int64_t bx = (stride + 255) / 256;
  if (bx < 1) bx = 1;
  hipLaunchKernelGGL(k_seg, dim3((unsigned)bx, (unsigned)P), dim3(256), 0, s, idx, stride, nnz,
                     P, d, ntiles_u, seg, status);
  return hipGetLastError();
}

hipError_t launch_update(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                         int32_t d, int32_t ntiles_u, const int32_t* idx, const float* val,
                         int64_t stride, const int32_t* nnz, int32_t P, const int32_t* seg,
                         float lr, float mu, float wd, int sparse_mode, int has_mom,
                         hipStream_t s) {
  const int32_t per_xcd = (ntiles_u + kXcds - 1) / kXcds;
  hipLaunchKernelGGL(k_update, dim3(per_xcd * kXcds), dim3(kUBlock), 0, s, tens, tile_first,
                     ntens, d, ntiles_u, per_xcd, idx, val, stride, nnz, P, seg, lr, mu, wd,
                     sparse_mode, has_mom);
  return hipGetLastError();
}

}  // namespace tkef

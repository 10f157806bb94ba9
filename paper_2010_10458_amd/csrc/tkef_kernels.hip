// gfx950 kernels for exact top-k sparsification with error feedback and the
// sparse aggregate + multi-tensor SGD update.
//
// Sparsify (Sec. 3.1 TopK operator, read as exactly k elements with ties to
// the lower position; Alg. 1 output: ascending indices and the values of x):
//   stream   x = g + r stored into r; 11-bit histogram of the magnitude key;
//            one 16-bit max-key summary per 32-element line
//   then a three-level radix select of the k-th largest key (11, 10 and 10
//   bits) that reads only the lines whose summary reaches the current key
//   class, and an ordered compaction of the selected (idx, val) with r[idx]
//   set to +0:
//   one group (global top-k):  collect, finish
//   per-tensor groups:         pick 1, gather, pick 2, hist3, pick 3,
//                              groupscan, emit
// For rho << 1 the data is streamed from HBM once; the later kernels touch a
// small fraction of it.
//
// Update (Alg. 2 accumulation of the gathered lists; Eq. (1) with optional
// weight decay and momentum):
//   seg      per worker, the first list entry of every update tile (the lists
//            are ascending, so tile boundaries are where idx >> shift grows)
//   update   per tile: LDS accumulation of all workers' entries of the tile,
//            then one pass applying the SGD step to that parameter range
#include <mutex>

#include <hip/hip_ext.h>
#include <hip/hip_fp16.h>
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

// Inclusive prefix sum over the 64 lanes of a wavefront: DPP row shifts
// (1, 2, 4, 8) within each row of 16 lanes, then the totals of the lower rows
// added from readlane.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  const uint32_t t0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t t1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t t2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = (int)(threadIdx.x & 63) >> 4;
  x += (row > 0 ? t0 : 0u) + (row > 1 ? t1 : 0u) + (row > 2 ? t2 : 0u);
  return x;
}

// Exclusive prefix sums of two values per thread over an NT-thread
// workgroup (wave scans, then the wave totals through LDS). wsum: 2 * NT / 64
// words of LDS. Returns the two prefixes; *total gets the two sums. Two
// barriers; the second lets the next call reuse wsum.
template <int NT>
__device__ __forceinline__ uint2 block_scan2(uint32_t a, uint32_t b, uint32_t* wsum,
                                             uint2* total) {
  constexpr int NW = NT / 64;
  const int tid = threadIdx.x, wid = tid >> 6;
  const uint32_t xa = wave_incl_scan(a), xb = wave_incl_scan(b);
  if ((tid & 63) == 63) {
    wsum[wid] = xa;
    wsum[NW + wid] = xb;
  }
  __syncthreads();
  uint32_t ba = 0u, bb = 0u, ta = 0u, tb = 0u;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t sa = wsum[i], sb = wsum[NW + i];
    ba += (i < wid) ? sa : 0u;
    bb += (i < wid) ? sb : 0u;
    ta += sa;
    tb += sb;
  }
  *total = make_uint2(ta, tb);
  __syncthreads();
  return make_uint2(ba + xa - a, bb + xb - b);
}

// Exclusive prefix sums of four values per thread (same scheme and barriers).
// wsum: 4 * NT / 64 words. pre[] and tot[] get the prefixes and the sums.
template <int NT>
__device__ __forceinline__ void block_scan4(const uint32_t (&v)[4], uint32_t* wsum,
                                            uint32_t (&pre)[4], uint32_t (&tot)[4]) {
  constexpr int NW = NT / 64;
  const int tid = threadIdx.x, wid = tid >> 6;
  uint32_t x[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) x[c] = wave_incl_scan(v[c]);
  if ((tid & 63) == 63) {
#pragma unroll
    for (int c = 0; c < 4; ++c) wsum[c * NW + wid] = x[c];
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    uint32_t b = 0u, t = 0u;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t sv = wsum[c * NW + i];
      b += (i < wid) ? sv : 0u;
      t += sv;
    }
    pre[c] = b + x[c] - v[c];
    tot[c] = t;
  }
  __syncthreads();
}

// One exclusive prefix sum over an NT-thread workgroup. wsum: NT / 64 words.
template <int NT>
__device__ __forceinline__ uint32_t block_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  constexpr int NW = NT / 64;
  const int tid = threadIdx.x, wid = tid >> 6;
  const uint32_t x = wave_incl_scan(v);
  if ((tid & 63) == 63) wsum[wid] = x;
  __syncthreads();
  uint32_t before = 0u, all = 0u;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t sv = wsum[i];
    before += (i < wid) ? sv : 0u;
    all += sv;
  }
  *total = all;
  __syncthreads();
  return before + x - v;
}

// Device-memory views of pointers that were read from memory (tile
// descriptors, LDS lists): loads and stores through them then use the global
// instructions, whose completion counter is not shared with LDS operations.
typedef __attribute__((address_space(1))) float gfloat;
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) v4f gv4f;
__device__ __forceinline__ const gfloat* gptr(const float* p) { return (const gfloat*)p; }
__device__ __forceinline__ gfloat* gptr(float* p) { return (gfloat*)p; }

// Loads the elements [e0, e0 + n) of one line (0 <= n <= kLine) of x into
// v[]; v[q] for q >= n is unspecified (callers mask by n).
__device__ __forceinline__ void load_line(const float* __restrict__ x, int e0, int n,
                                          float (&v)[kLine]) {
  const float* p = x + e0;
  if (n == kLine && (reinterpret_cast<uintptr_t>(p) & 15u) == 0) {
    const gv4f* p4 = (const gv4f*)p;
#pragma unroll
    for (int q = 0; q < kLine / 4; ++q) {
      const v4f f = p4[q];
      v[4 * q + 0] = f.x;
      v[4 * q + 1] = f.y;
      v[4 * q + 2] = f.z;
      v[4 * q + 3] = f.w;
    }
  } else if (n > 0) {
    const gfloat* g = gptr(p);  // clamped indices: every load stays inside the line
#pragma unroll
    for (int q = 0; q < kLine; ++q) v[q] = g[min(q, n - 1)];
  }
}

// v[j] for a j that differs between lanes: a tree of selects on the bits of
// j, written as bit arithmetic (a select of two array elements would be
// turned into an indexed access, which moves v out of registers).
__device__ __forceinline__ uint32_t sel_bits(uint32_t m, uint32_t a, uint32_t b) {
  return a ^ ((a ^ b) & m);  // m == 0: a, m == ~0: b
}
__device__ __forceinline__ float pick_elem(const float (&v)[kLine], int j) {
  static_assert(kLine == 32, "five select levels");
  uint32_t a[16], b[8], c[4], d[2];
  const uint32_t m0 = 0u - (uint32_t)(j & 1), m1 = 0u - (uint32_t)((j >> 1) & 1),
                 m2 = 0u - (uint32_t)((j >> 2) & 1), m3 = 0u - (uint32_t)((j >> 3) & 1),
                 m4 = 0u - (uint32_t)((j >> 4) & 1);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    a[i] = sel_bits(m0, __float_as_uint(v[2 * i]), __float_as_uint(v[2 * i + 1]));
#pragma unroll
  for (int i = 0; i < 8; ++i) b[i] = sel_bits(m1, a[2 * i], a[2 * i + 1]);
#pragma unroll
  for (int i = 0; i < 4; ++i) c[i] = sel_bits(m2, b[2 * i], b[2 * i + 1]);
#pragma unroll
  for (int i = 0; i < 2; ++i) d[i] = sel_bits(m3, c[2 * i], c[2 * i + 1]);
  return __uint_as_float(sel_bits(m4, d[0], d[1]));
}

// Values on the wire: binary32, or binary16 rounded to nearest even (Sec. 5.3
// sends FP16 elements). val16 selects the format of the value array.
__device__ __forceinline__ void put_val(void* out, size_t pos, float x, int val16) {
  if (val16) reinterpret_cast<uint16_t*>(out)[pos] = __half_as_ushort(__float2half_rn(x));
  else reinterpret_cast<float*>(out)[pos] = x;
}
__device__ __forceinline__ float get_val(const void* in, size_t pos, int val16) {
  return val16 ? __half2float(__ushort_as_half(reinterpret_cast<const uint16_t*>(in)[pos]))
               : reinterpret_cast<const float*>(in)[pos];
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
// compact window of memory. g and r are read and x is written with
// non-temporal accesses: each element is touched once, and normal stores,
// although a little faster for the stream alone, leave dirty lines whose
// write-back slows the kernels that follow. Each workgroup keeps an LDS
// histogram and adds it to one of `nslots` copies of its group's global
// histogram when the group changes and at the end; the copies spread the
// atomics of many workgroups over many addresses.
constexpr int kQuarter = kStreamUnit;
constexpr int kQV = kQuarter / (4 * kBlock);  // float4 of each array per thread per unit
static_assert(kQV * 4 * kBlock == kQuarter && kTile % kQuarter == 0, "stream unit shape");

// Non-temporal 16-byte load / store through a global-memory view.
__device__ __forceinline__ float4 load_nt4(const float4* p) {
  const v4f t = __builtin_nontemporal_load((const gv4f*)p);
  return make_float4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ void store_nt4(float4* p, float4 v) {
  const v4f t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, (gv4f*)p);
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

// clear: clear_words words of the scratch that only later kernels of the
// execution use (zeroed here for them; nothing in this kernel reads them).
__global__ __launch_bounds__(kBlock) void k_stream(const TileDesc* __restrict__ tiles,
                                                   int32_t ntiles, uint32_t* __restrict__ hist1,
                                                   int nslots, uint16_t* __restrict__ summ,
                                                   uint32_t* __restrict__ status,
                                                   uint32_t* __restrict__ clear,
                                                   int64_t clear_words) {
  __shared__ uint32_t h[kH1Bins];
  __shared__ uint32_t nanflag;
  const int tid = threadIdx.x;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + tid; i < clear_words;
       i += (int64_t)gridDim.x * kBlock)
    clear[i] = 0u;
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
      // kQV float4 of g and of r per thread, all loads in flight together; a
      // line is 8 consecutive lanes
      const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
      float4* __restrict__ r4 = reinterpret_cast<float4*>(r);
      float4 a[kQV], b[kQV];
#pragma unroll
      for (int v = 0; v < kQV; ++v) a[v] = load_nt4(g4 + v * kBlock + tid);
#pragma unroll
      for (int v = 0; v < kQV; ++v) b[v] = load_nt4(r4 + v * kBlock + tid);
#pragma unroll
      for (int v = 0; v < kQV; ++v) {
        float4 x;
        uint32_t m = add_quad(a[v], b[v], x, h);
        store_nt4(r4 + v * kBlock + tid, x);
        tmax = max(tmax, m);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        m = max(m, (uint32_t)__shfl_xor((int)m, 4));
        if ((tid & 7) == 0) sq[(v * kBlock + tid) >> 3] = (uint16_t)(m >> 16);
      }
    } else {
      // partial or misaligned quarter: element by element (coalesced 4-byte
      // accesses), every load issued before the first use so the quarter
      // costs one memory latency. Element e = q * kBlock + tid: a wavefront's
      // 64 lanes hold two whole lines, so a line's maximum key is a
      // reduction over 32 lanes (lanes past the end contribute 0); the
      // summary of a line without elements is not written.
      constexpr int kPer = kQuarter / kBlock;
      float gv[kPer], rv[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        gv[q] = (e < len) ? __builtin_nontemporal_load(gptr(g) + e) : 0.0f;
        rv[q] = (e < len) ? __builtin_nontemporal_load(gptr(r) + e) : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        uint32_t k = 0u;
        if (e < len) {
          const float x = gv[q] + rv[q];
          __builtin_nontemporal_store(x, gptr(r) + e);
          k = mag_key(x);
          atomicAdd(&h[k >> kH1Shift], 1u);
          tmax = max(tmax, k);
        }
        k = max(k, (uint32_t)__shfl_xor((int)k, 1));
        k = max(k, (uint32_t)__shfl_xor((int)k, 2));
        k = max(k, (uint32_t)__shfl_xor((int)k, 4));
        k = max(k, (uint32_t)__shfl_xor((int)k, 8));
        k = max(k, (uint32_t)__shfl_xor((int)k, 16));
        if ((tid & (kLine - 1)) == 0 && e < len) sq[e / kLine] = (uint16_t)(k >> 16);
      }
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
// PER consecutive bins, summed over the histogram's NSLOT copies with 16-byte
// loads that are all in flight together.
template <int PER, int NSLOT>
__global__ __launch_bounds__(kBlock) void k_pick(int level, const GroupDesc* __restrict__ groups,
                                                 GroupState* __restrict__ st,
                                                 const uint32_t* __restrict__ hist) {
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
  const uint32_t* __restrict__ hg = hist + (size_t)g * NSLOT * nbins + lo;
  uint4 v[NSLOT][PER / 4];
#pragma unroll
  for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
    for (int q = 0; q < PER / 4; ++q)
      v[sl][q] = reinterpret_cast<const uint4*>(hg + (size_t)sl * nbins)[q];
  uint32_t c[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) c[j] = 0u;
#pragma unroll
  for (int sl = 0; sl < NSLOT; ++sl) {
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
      c[4 * q + 0] += v[sl][q].x;
      c[4 * q + 1] += v[sl][q].y;
      c[4 * q + 2] += v[sl][q].z;
      c[4 * q + 3] += v[sl][q].w;
    }
  }
  uint32_t sum = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) sum += c[j];
  uint32_t total;
  const uint32_t excl = block_scan<kBlock>(sum, part, &total);
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
// Selection kernels after the stream.
//
// They run as at most kSMaxGroups workgroups of kSBlock threads (collect and
// finish: NT threads, see below), each thread owning `lpt` consecutive
// summary lines (or, in the per-tensor emit and hist3, a run of the compacted
// candidate list). A candidate is encoded as (tile << 13) | position-in-tile,
// in the per-tensor list together with the bits of x.
//
// The per-tensor path places its ordered output with a prefix of
// per-workgroup counts: each workgroup publishes its count in a flag word
// (bit 63 = valid) and then reads the words of all lower-numbered
// workgroups. It waits only on workgroups dispatched before it (workgroups
// start in order of their number), which publish without waiting on
// anything, so the wait ends; it is still bounded (kSpinLimit polls per
// word), after which TKEF_STATUS_TIMEOUT is recorded and the workgroup writes
// no output that depends on the prefix. Flag words are cleared before every
// execution.
constexpr int kSBlock = 1024;
constexpr int kSWaves = kSBlock / 64;
// collect and finish (one selection group) run kCBlockSmall threads per
// workgroup, with more lines per thread, for inputs of up to kCSmallLines
// summary lines: their per-thread steps (summaries, scans, bins) are short
// instruction runs over every thread of a region, so fewer threads per
// compute unit finish them sooner. Larger inputs take kSBlock threads, whose
// regions hold more flagged lines, so each thread walks fewer of them;
// except dense selections (k >= d / kCDenseDiv), whose many flagged lines
// are walked faster by two half-size workgroups per compute unit, one
// loading its lines while the other works through its own (110 M
// elements: 375 against 387 us at rho = 0.01, 342 against 347 at 0.007, even
// at 0.005, 8-10 us slower at 0.002-0.004), as long as the half-size
// regions number at most kCDenseMaxGroups: every finish workgroup's work
// grows with the number of regions (340 M elements, 1,297 regions: 1,372
// against 1,310 us at rho = 0.01).
constexpr int kCBlockSmall = 512;
constexpr int64_t kCSmallLines = (int64_t)256 * kCBlockSmall * 8;
constexpr int64_t kCDenseDiv = 160;
constexpr int64_t kCDenseMaxGroups = 512;
constexpr int kSMaxGroups = 4096;
constexpr int kSMaxLpt = 16;     // lines per thread at most
static_assert(kLinesPerTile % kSMaxLpt == 0, "a thread's lines lie in one tile");
constexpr int kCandShift = 13;   // log2(kTile)
static_assert((1 << kCandShift) == kTile, "candidate encoding");
static_assert((int64_t)kSMaxGroups * kSBlock * kSMaxLpt >= kMaxTiles * kLinesPerTile &&
              (int64_t)kSMaxGroups * kCBlockSmall * kSMaxLpt >= kCSmallLines,
              "the selection grids cover every tile of a list");
constexpr uint64_t kFlagValid = 1ull << 63, kFlagVal = (1ull << 63) - 1;
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kStage = 8;       // candidates a thread stages in LDS
constexpr int kEmitLdsGroups = kSBlock;  // group bases k_emit forms itself (8 KB of LDS)
constexpr int kGStage = 24;     // ... in gather (dense per-tensor selections; 144 KB)

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

__device__ __forceinline__ uint32_t sblock_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  return block_scan<kSBlock>(v, wsum, total);
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
// workgroups numbered below it (uniform in the workgroup).
//
// The wait relies on the dispatcher starting a grid's workgroups in order of
// their number, so that every workgroup numbered below a waiting one has
// started and will publish its count; the callers' grids are also sized so
// that all their workgroups are resident at once. Each wait is bounded
// (kSpinLimit sleeps): a workgroup that gives up sets TKEF_STATUS_TIMEOUT,
// and *ok = false tells the caller that the prefix is incomplete, so that it
// writes nothing that depends on it.
__device__ uint64_t group_prefix(uint64_t* __restrict__ flags, uint64_t mine, uint64_t* red,
                                 uint32_t* __restrict__ status, bool* ok) {
  const int tid = threadIdx.x;
  const int w = blockIdx.x;
  if (tid == 0) flag_store(&flags[w], kFlagValid | mine);
  uint64_t v = 0;
  bool gave_up = false;
  for (int j = tid; j < w && !gave_up; j += kSBlock) {
    uint64_t f = flag_load(&flags[j]);
    uint32_t spins = 0;
    while (!(f & kFlagValid)) {
      if (++spins > kSpinLimit) {
        gave_up = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      f = flag_load(&flags[j]);
    }
    v += f & kFlagVal;
  }
  const bool any = __syncthreads_or(gave_up ? 1 : 0) != 0;
  if (any && tid == 0 && status) atomicOr(status, TKEF_STATUS_TIMEOUT);
  *ok = !any;
  return sblock_sum_u64(v, red);
}

// Within one NT-thread workgroup: the bin of an NB-bin histogram, held in
// NSLOT copies NB words apart (summed), where the running count from the
// highest bin reaches `need`. Thread t owns the NB / NT bins from
// NB - 1 - t NB / NT downwards, read as one 8- or 16-byte load per copy (hist
// 16-byte aligned); all its loads are issued before the first is used. res[] (LDS): bin, count above it, count in it; all zero if no bin
// does (need == 0 or above the total). Exactly one thread writes res[], after
// the scan's barriers (so every reader of an earlier result is done); ends
// with a barrier.
template <int NT, int NB, int NSLOT>
__device__ __forceinline__ void block_pick(const uint32_t* __restrict__ hist, uint32_t need,
                                           uint32_t* wsum, uint32_t* res) {
  constexpr int BPT = NB / NT;
  static_assert(BPT >= 1 && BPT * NT == NB, "whole bins per thread");
  static_assert(BPT == 1 || BPT == 2 || BPT == 4, "one load per copy");
  const int tid = threadIdx.x;
  const int top = NB - 1 - BPT * tid;
  uint32_t v[NSLOT][BPT];  // v[sl][b]: bin top - b
#pragma unroll
  for (int sl = 0; sl < NSLOT; ++sl) {
    const uint32_t* src = hist + (size_t)sl * NB + (top - (BPT - 1));
    if constexpr (BPT == 4) {
      const uint4 q = *reinterpret_cast<const uint4*>(src);
      v[sl][0] = q.w;
      v[sl][1] = q.z;
      v[sl][2] = q.y;
      v[sl][3] = q.x;
    } else if constexpr (BPT == 2) {
      const uint2 q = *reinterpret_cast<const uint2*>(src);
      v[sl][0] = q.y;
      v[sl][1] = q.x;
    } else {
      v[sl][0] = src[0];
    }
  }
  uint32_t c[BPT], sum = 0u;
#pragma unroll
  for (int b = 0; b < BPT; ++b) {
    c[b] = 0u;
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) c[b] += v[sl][b];
    sum += c[b];
  }
  uint32_t total;
  uint32_t run = block_scan<NT>(sum, wsum, &total);
#pragma unroll
  for (int b = 0; b < BPT; ++b) {
    if (run < need && need <= run + c[b]) {
      res[0] = (uint32_t)(top - b);
      res[1] = run;
      res[2] = c[b];
    }
    run += c[b];
  }
  if ((need == 0u || need > total) && tid == NT - 1) {
    res[0] = 0u;
    res[1] = 0u;
    res[2] = 0u;
  }
  __syncthreads();
}

// The thread's `lpt` consecutive summary lines starting at line l0. lpt is a
// power of two from 4 up to kSMaxLpt and divides kLinesPerTile, so all of
// them lie in one tile. flagged() gives the lines whose summary reaches
// thr(group). Lines past a tile's elements keep the summary 0 that bind
// writes (the stream never writes them), so they are flagged only for
// thr < 2^16, and hold no elements then. Summaries (two per register) and the
// descriptor are fetched together up front.
struct LineSpan {
  static constexpr int MAXL = kSMaxLpt;
  static_assert(MAXL % 4 == 0 && MAXL <= 32, "line mask width");
  int tile, e0, lim;  // tile, position of the first line's first element, lines held
  TileDesc t;
  uint32_t sp[MAXL / 2];

  __device__ __forceinline__ void load(const TileDesc* __restrict__ tiles,
                                       const uint16_t* __restrict__ summ, int64_t nlines,
                                       int64_t l0, int lpt) {
    const bool has = l0 < nlines;  // nlines is a multiple of kLinesPerTile
    tile = has ? (int)(l0 / kLinesPerTile) : 0;
    e0 = (int)(l0 % kLinesPerTile) * kLine;
    // four summaries per 8-byte load (l0 and lpt are multiples of 4)
#pragma unroll
    for (int c = 0; c < MAXL / 4; ++c) {
      uint2 v = make_uint2(0u, 0u);
      if (has && 4 * c < lpt) v = *reinterpret_cast<const uint2*>(summ + l0 + 4 * c);
      sp[2 * c] = v.x;
      sp[2 * c + 1] = v.y;
    }
    t = tiles[tile];
    lim = has ? lpt : 0;
  }
  __device__ __forceinline__ int e0_of(int q) const { return e0 + q * kLine; }
  template <typename Thr>
  __device__ __forceinline__ uint32_t flagged(Thr thr) const {
    const uint32_t th = thr(t.group) >> 16;
    uint32_t m = 0u;
#pragma unroll
    for (int q = 0; q < MAXL; ++q) {
      const uint32_t sv = (sp[q >> 1] >> (16 * (q & 1))) & 0xFFFFu;
      m |= (q < lim && sv >= th) ? (1u << q) : 0u;
    }
    return m;
  }
};

// For every element of the flagged lines in `mask`, in position order, for
// which hit(group, key) holds: f(tile, TileDesc, e, x, key). The hit test runs
// over all 32 elements of a line at once; the hits are then visited one by
// one, each taken from the line already in registers.
template <typename Hit, typename F>
__device__ __forceinline__ void walk_mask(const LineSpan& ls, uint32_t mask, Hit hit, F f) {
#pragma unroll 1
  while (mask) {
    const int q = __ffs(mask) - 1;
    mask &= mask - 1u;
    const TileDesc& t = ls.t;
    const int e0 = ls.e0_of(q), n = max(0, min(kLine, t.len - e0));
    float v[kLine];
    load_line(t.r, e0, n, v);
    uint32_t hm = 0u;
#pragma unroll
    for (int j = 0; j < kLine; ++j)
      hm |= (j < n && hit(t.group, mag_key(v[j]))) ? (1u << j) : 0u;
    const int tile = ls.tile;
#pragma unroll 1
    while (hm) {
      const int j = __ffs(hm) - 1;
      hm &= hm - 1u;
      const float x = pick_elem(v, j);
      f(tile, t, e0 + j, x, mag_key(x));
    }
  }
}

// Calls f(tile, TileDesc, e, x, key) for candidates [cb, ce), in order. A
// candidate is {(tile << 13) | position-in-tile, bits of x}; four are taken
// at a time, their entries and then their tile descriptors fetched together.
template <typename F>
__device__ __forceinline__ void walk_cands(const TileDesc* __restrict__ tiles, int32_t ntiles,
                                           const uint2* __restrict__ cand, uint32_t cb,
                                           uint32_t ce, F f) {
#pragma unroll 1
  for (uint32_t j = cb; j < ce; j += 4) {
    uint2 q[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) q[c] = cand[min(j + (uint32_t)c, ce - 1u)];  // clamped
    TileDesc t[4];
#pragma unroll
    for (int c = 0; c < 4; ++c)  // an entry never names a tile >= ntiles; clamped anyway
      t[c] = tiles[min((int)(q[c].x >> kCandShift), ntiles - 1)];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int tile = (int)(q[c].x >> kCandShift);
      const int e = (int)(q[c].x & (kTile - 1));
      if (j + (uint32_t)c >= ce || tile >= ntiles || e >= t[c].len) continue;
      const float x = __uint_as_float(q[c].y);
      f(tile, t[c], e, x, mag_key(x));
    }
  }
}

// ---------------------------------------------------------------------------
// One selection group (top-k over all tensors together): collect, finish.
//
// Workgroup w of either kernel (NT threads) owns the region of summary lines
// [w * NT * lpt, (w + 1) * NT * lpt), lpt consecutive lines per thread. No workgroup waits on another: the ordered output is placed from
// small per-region counts that collect leaves behind.
//
// collect makes the level-1 pick (bin B1 of the k-th largest key) itself from
// the slotted histogram. The region's flagged lines (summary >= B1 << 20) are
// listed in LDS in position order and read one line per thread, all in one
// round. It writes
//   rcand[w]    the candidates (key >= B1 << 20) in position order, as
//               {global index, bits of x, address of the residual element};
//   rband[w]    the keys of the band members (key >> 20 == B1), ordered by
//               level-2 bin (key bits 19..10) from the top;
//   rsuf[w][b]  band members of the region in level-2 bins above b (written
//               when the region has band members);
//   rbin[b][w]  the first kPerBin keys of rband[w] in level-2 bin b (slots
//               beyond the bin's count are left as they were);
//   rcnt[w]     {candidates | (rcand incomplete) << 31,
//                band members | (band not stored) << 31}, counts exact;
//   hist2       += the region's level-2 histogram.
// A region with more than rcap candidates leaves rcand incomplete; one with
// more than kBandCap band members keeps the rest in rbtmp[w] (global
// scratch) until they are placed; one with more than rcap stores no band keys
// (rband, rbin), and finish then reads that region's lines instead.
//
// finish makes the level-2 pick (bin B2) from hist2, builds the level-3
// histogram in LDS from the band members in bin B2 of all regions (from rbin
// and the counts in rsuf; from rband when a region has more than kPerBin) and
// picks the exact threshold key T and the number of elements equal to T to
// keep. The elements above T in the regions before
// its own are the non-band candidates, the band members above bin B2 and the
// bin-B2 members above T; the elements equal to T are bin-B2 members. From
// these counts workgroup w places its region's selection.
constexpr int kOvWords = kSMaxGroups / 32;
constexpr int kFlCap = 4096;     // flagged lines listed in LDS at a time
constexpr int kBandCap = 4096;   // band members of a region kept in LDS
constexpr int kC2Cap = 4096;     // level-2 class members kept in LDS by finish
static_assert(kPerBin == 4, "rbin entries are read as one uint4");
static_assert(kSMaxGroups <= 65536, "region numbers fit 16 bits");

// (The sizes come last among the arguments: they are used at the start, so
// both cache lines of the argument block are fetched then, and later reloads
// of the pointers hit.)
template <int NT>
__global__ __launch_bounds__(NT, 4) void k_collect(
    const TileDesc* __restrict__ tiles, const GroupDesc* __restrict__ groups,
    GroupState* __restrict__ st, const uint32_t* __restrict__ hist1,
    const uint16_t* __restrict__ summ, uint32_t* __restrict__ hist2,
    uint32_t* __restrict__ rbin, uint4* __restrict__ rcand, uint32_t* __restrict__ rband,
    uint32_t* __restrict__ rbtmp, uint32_t* __restrict__ rsuf, uint2* __restrict__ rcnt,
    uint32_t rcap, int lpt, int64_t nlines) {
  __shared__ uint32_t h[kH2Bins];
  __shared__ uint32_t hoff[kH2Bins];
  __shared__ uint32_t wsum[2 * (NT / 64)];
  __shared__ uint32_t res[3];
  __shared__ float* lptr[kFlCap];        // flagged lines: first element
  __shared__ uint32_t lgidx[kFlCap];     // global index of the first element
  __shared__ uint8_t lnum[kFlCap];       // elements in the line
  __shared__ uint32_t bandk[kBandCap];
  __shared__ uint32_t nband;
  const int tid = threadIdx.x, w = blockIdx.x;
  for (int i = tid; i < kH2Bins; i += NT) h[i] = 0u;
  if (tid == 0) nband = 0u;

  // summaries of this thread's lines (independent of the pick), then the
  // level-1 pick, whose barriers also publish the cleared LDS
  LineSpan ls;
  ls.load(tiles, summ, nlines, ((int64_t)w * NT + tid) * lpt, lpt);
  __builtin_amdgcn_sched_barrier(0);  // keep those loads ahead of the histogram's
  const uint32_t k = groups[0].k;
  block_pick<NT, kH1Bins, kSlotsOne>(hist1, k, wsum, res);
  const uint32_t B1 = res[0];
  const uint32_t above1 = res[1];
  const uint32_t lo = B1 << kH1Shift;

  // flagged lines in position order: thread order, then line order
  const uint32_t mask = ls.flagged([&](int) -> uint32_t { return lo; });
  uint32_t F;
  const uint32_t fex = block_scan<NT>((uint32_t)__popc(mask), wsum, &F);
  uint32_t cw = 0u;   // candidates so far (workgroup-uniform)
  bool fits = true;   // workgroup-uniform
  uint4* __restrict__ cdst = rcand + (size_t)w * rcap;
#pragma unroll 1
  for (uint32_t c0 = 0; c0 < F; c0 += kFlCap) {
    uint32_t m = mask, rank = fex;
#pragma unroll 1
    while (m) {
      const int q = __ffs(m) - 1;
      m &= m - 1u;
      if (rank >= c0 && rank < c0 + (uint32_t)kFlCap) {
        const TileDesc& t = ls.t;
        const int e0 = ls.e0_of(q);
        lptr[rank - c0] = t.r + e0;
        lgidx[rank - c0] = (uint32_t)(t.gstart + e0);
        lnum[rank - c0] = (uint8_t)max(0, min(kLine, t.len - e0));
      }
      ++rank;
    }
    __syncthreads();
    const uint32_t nl = min((uint32_t)kFlCap, F - c0);
#pragma unroll 1
    for (uint32_t b0 = 0; b0 < nl; b0 += NT) {
      const uint32_t i = b0 + tid;
      float v[kLine];
      uint32_t hm = 0u, bm = 0u, gidx0 = 0u;  // candidates, band members of the line
      float* rp = nullptr;
      if (i < nl) {
        gidx0 = lgidx[i];
        rp = lptr[i];
        const int n = lnum[i];
        load_line(rp, 0, n, v);
#pragma unroll
        for (int j = 0; j < kLine; ++j) {
          const uint32_t key = mag_key(v[j]);
          hm |= (j < n && key >= lo) ? (1u << j) : 0u;
          bm |= (j < n && (key >> kH1Shift) == B1) ? (1u << j) : 0u;
        }
      }
      {
        // band slots: one atomic per wavefront, shared out by a wave scan
        const uint32_t bc = (uint32_t)__popc(bm);
        const uint32_t incl = wave_incl_scan(bc);
        const uint32_t wtot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
        uint32_t wbase = 0u;
        if ((tid & 63) == 63 && wtot) wbase = atomicAdd(&nband, wtot);
        wbase = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 63);
        uint32_t slot = wbase + incl - bc;
#pragma unroll 1
        for (uint32_t m2 = bm; m2; m2 &= m2 - 1u, ++slot) {
          const uint32_t key = mag_key(pick_elem(v, __ffs(m2) - 1));
          atomicAdd(&h[(key >> kH2Shift) & (kH2Bins - 1)], 1u);
          if (slot < (uint32_t)kBandCap) bandk[slot] = key;
          else if (slot < rcap) rbtmp[(size_t)w * rcap + slot] = key;
        }
      }
      uint32_t tot;
      const uint32_t ex = block_scan<NT>((uint32_t)__popc(hm), wsum, &tot);
      if (cw + tot > rcap) fits = false;
      if (fits && hm) {
        uint4* __restrict__ dst = cdst + cw + ex;
#pragma unroll 1
        for (uint32_t m2 = hm; m2; m2 &= m2 - 1u, ++dst) {
          const int j = __ffs(m2) - 1;
          const uint64_t a = reinterpret_cast<uint64_t>(rp + j);
          *dst = make_uint4(gidx0 + (uint32_t)j, __float_as_uint(pick_elem(v, j)), (uint32_t)a,
                            (uint32_t)(a >> 32));
        }
      }
      cw += tot;
    }
    // the line list is refilled for the next chunk (skipped after the last)
    if (c0 + (uint32_t)kFlCap < F) __syncthreads();
  }

  // band members by level-2 bin from the top (thread t owns the kB2 bins
  // from 1023 - kB2 t downwards): sorted into rband[w], and the first
  // kPerBin of each bin also into rbin
  constexpr int kB2 = kH2Bins / NT;
  const int top = kH2Bins - 1 - kB2 * tid;
  uint32_t cb[kB2], ab[kB2], csum = 0u;
#pragma unroll
  for (int b = 0; b < kB2; ++b) {
    cb[b] = h[top - b];
    csum += cb[b];
  }
  uint32_t bw;
  uint32_t above = block_scan<NT>(csum, wsum, &bw);
  const bool band_ok = bw <= rcap;  // the band fits rband[w] (and rbtmp[w])
#pragma unroll
  for (int b = 0; b < kB2; ++b) {
    ab[b] = above;
    h[top - b] = above;     // from here on: the bin's next slot in rband[w]
    hoff[top - b] = above;  // the bin's first slot
    above += cb[b];
  }
  __syncthreads();
#pragma unroll
  for (int b = 0; b < kB2; ++b) {
    if (cb[b]) atomicAdd(&hist2[top - b], cb[b]);
    if (bw) rsuf[(size_t)w * kH2Bins + top - b] = ab[b];
  }
  uint32_t* __restrict__ dst = rband + (size_t)w * rcap;
  auto place = [&](uint32_t key) {
    const uint32_t b2 = (key >> kH2Shift) & (kH2Bins - 1);
    const uint32_t slot = atomicAdd(&h[b2], 1u);
    dst[slot] = key;
    const uint32_t rank = slot - hoff[b2];
    if (rank < (uint32_t)kPerBin) rbin[((size_t)b2 * gridDim.x + w) * kPerBin + rank] = key;
  };
  if (band_ok) {
    // the first kBandCap from LDS, the rest (a dense selection) from the
    // region's scratch in rbtmp, written before the barriers above. Two loops:
    // a read through a pointer that may point to either would be a flat load,
    // which waits for every global store and atomic issued above.
    const uint32_t nlds = min(bw, (uint32_t)kBandCap);
    for (uint32_t j = tid; j < nlds; j += NT) place(bandk[j]);
    const uint32_t* __restrict__ tmp = rbtmp + (size_t)w * rcap;
    for (uint32_t j = (uint32_t)kBandCap + tid; j < bw; j += NT) place(tmp[j]);
  }
  if (tid == 0)
    rcnt[w] = make_uint2(cw | ((fits ? 0u : 1u) << 31), bw | ((band_ok ? 0u : 1u) << 31));
  if (w == 0 && tid == 0) {  // the level-1 result
    GroupState s;
    s.need = (above1 < k) ? k - above1 : 0u;
    s.prefix = B1;
    s.T = 0xFFFFFFFFu;
    s.n_eq = 0u;
    st[0] = s;
  }
}

// Calls f(key) for the level-2 class members (band members in bin B2) of the
// stored regions among [0, wlim), reading them again from rband. Regions are
// taken NT at a time and their members spread over the workgroup through
// a scan of the per-region counts. off, abv: NT words of LDS each.
// Uniform in the workgroup.
template <int NT, typename F>
__device__ __forceinline__ void for_class2(int wlim, uint32_t B2, uint32_t rcap,
                                           const uint2* __restrict__ rcnt,
                                           const uint32_t* __restrict__ rsuf,
                                           const uint32_t* __restrict__ rband, uint32_t* off,
                                           uint32_t* abv, uint32_t* wsum, F f) {
  const int tid = threadIdx.x;
#pragma unroll 1
  for (int r0 = 0; r0 < wlim; r0 += NT) {
    const int r = r0 + tid;
    uint32_t above = 0u, at = 0u;
    if (r < wlim) {
      const uint2 cnt = rcnt[r];
      const uint32_t bw = cnt.y & 0x7FFFFFFFu;
      if (bw && !(cnt.y >> 31)) {
        const uint32_t* sr = rsuf + (size_t)r * kH2Bins;
        above = sr[B2];
        at = (B2 ? sr[B2 - 1] : bw) - above;
      }
    }
    uint32_t tot;
    const uint32_t ex = block_scan<NT>(at, wsum, &tot);
    off[tid] = ex;
    abv[tid] = above;
    __syncthreads();
#pragma unroll 1
    for (uint32_t j = tid; j < tot; j += NT) {
      int a = 0, b = NT - 1;  // the last region slot with off <= j holds member j
      while (a < b) {
        const int m = (a + b + 1) >> 1;
        if (off[m] <= j) a = m; else b = m - 1;
      }
      f(rband[(size_t)(r0 + a) * rcap + abv[a] + (j - off[a])]);
    }
    __syncthreads();
  }
}

// (Four waves per SIMD: two 512-thread workgroups, or one of 1,024 threads,
// per compute unit, so that up to 512 regions are all resident at once; at
// 129 registers the 512-thread shape fitted one per compute unit and a
// grid of 424 regions ran in two rounds.)
template <int NT>
__global__ __launch_bounds__(NT, 4) void k_finish(
    const TileDesc* __restrict__ tiles, const GroupDesc* __restrict__ groups,
    const GroupState* __restrict__ st, const uint16_t* __restrict__ summ, int64_t nlines,
    int lpt, uint32_t rcap, const uint32_t* __restrict__ hist2,
    const uint32_t* __restrict__ rbin, const uint4* __restrict__ rcand,
    const uint32_t* __restrict__ rband,
    const uint32_t* __restrict__ rsuf, const uint2* __restrict__ rcnt,
    int32_t* __restrict__ idx_out, void* __restrict__ val_out, int val16,
    uint32_t* __restrict__ clear_next, int64_t clear_words, uint32_t* __restrict__ ticket,
    uint64_t* __restrict__ rzr) {
  __shared__ __align__(16) uint32_t h[kH3Bins];
  __shared__ uint32_t wsum[4 * (NT / 64)];
  __shared__ uint32_t res[3];
  __shared__ uint32_t off[NT], abv[NT];
  __shared__ uint32_t ovbits[kOvWords];  // regions whose band keys were not stored
  __shared__ uint32_t c2bits[kOvWords];  // ... of them, those holding level-2 class members
  __shared__ uint32_t c2key[kC2Cap];     // level-2 class members of the stored regions
  __shared__ uint16_t c2reg[kC2Cap];     // ... and their regions
  __shared__ uint32_t n2;
  __shared__ uint32_t any_unstored, last;
  constexpr int kRegPerThread = kSMaxGroups / NT;
  const int tid = threadIdx.x, w = blockIdx.x, G = gridDim.x;
  for (int i = tid; i < kH3Bins; i += NT) h[i] = 0u;
  for (int i = tid; i < kOvWords; i += NT) {
    ovbits[i] = 0u;
    c2bits[i] = 0u;
  }
  if (tid == 0) {
    n2 = 0u;
    any_unstored = 0u;
  }

  // fetched together: level-1 state, this region's counts and first
  // candidate, every region's counts (and, in the pick, the level-2 histogram)
  const GroupState s0 = st[0];
  const uint32_t k = groups[0].k;
  const uint2 mine = rcnt[w];
  const bool own_ov = (mine.x >> 31) != 0u;
  const uint4* __restrict__ mc = rcand + (size_t)w * rcap;
  // A region with more stored candidates than threads (dense selections)
  // takes them in rounds, candidate j on thread j % NT, so that a
  // wavefront's loads and output stores fall on consecutive entries;
  // otherwise each thread has at most one. (A region that stored its
  // candidates also stored its band, which they include: it never defers
  // its residual zeros, below.)
  const bool rounds = !own_ov && mine.x > (uint32_t)NT;
  uint32_t cb = 0u, ce = 0u;
  if (!own_ov && !rounds) {
    cb = min(mine.x, (uint32_t)tid);
    ce = min(mine.x, cb + 1u);
  }
  const uint4 v0 = (cb < ce || rounds) ? mc[rounds ? (uint32_t)tid : cb]
                                       : make_uint4(0u, 0u, 0u, 0u);
  uint2 cr[kRegPerThread];
#pragma unroll
  for (int q = 0; q < kRegPerThread; ++q) {
    const int r = q * NT + tid;
    cr[q] = make_uint2(0u, 0u);
    if (q * NT < G && r < G) cr[q] = rcnt[r];
  }

  // level 2 (the pick's barriers also publish the cleared LDS above)
  block_pick<NT, kH2Bins, 1>(hist2, s0.need, wsum, res);
  const uint32_t B2 = res[0];
  const uint32_t need2 = (res[1] < s0.need) ? s0.need - res[1] : 0u;
  const uint32_t cls21 = (s0.prefix << 10) | B2;

  // The level-2 class (band members in bin B2) of every region, fetched with
  // the counts that place it: per region, bw band members, `above` of them
  // in bins above B2 and `at` in bin B2, whose first kPerBin keys are in
  // rbin. gtb: this thread's share of the elements above T before region w.
  uint32_t gtb = 0u;
  bool slow = false;  // some region has more than kPerBin class-2 members
#pragma unroll
  for (int q = 0; q < kRegPerThread; ++q) {
    if (q * NT >= G) break;
    const int r = q * NT + tid;
    if (r >= G) continue;
    const uint32_t bw = cr[q].y & 0x7FFFFFFFu;
    const bool ov = (cr[q].y >> 31) != 0u;
    if (ov) {
      atomicOr(&ovbits[r >> 5], 1u << (r & 31));
      any_unstored = 1u;
    }
    if (!bw) {
      if (r < w) gtb += cr[q].x & 0x7FFFFFFFu;
      continue;
    }
    const uint32_t* sr = rsuf + (size_t)r * kH2Bins;
    const uint32_t above = sr[B2];
    const uint32_t at = (B2 ? sr[B2 - 1] : bw) - above;
    const uint4 e = *reinterpret_cast<const uint4*>(rbin + ((size_t)B2 * G + r) * kPerBin);
    if (r < w) gtb += (cr[q].x & 0x7FFFFFFFu) - bw + above;
    if (ov) {
      if (at) atomicOr(&c2bits[r >> 5], 1u << (r & 31));  // its lines are walked below
      continue;
    }
    if (at > (uint32_t)kPerBin) {
      slow = true;
      continue;
    }
    const uint32_t ek[4] = {e.x, e.y, e.z, e.w};
#pragma unroll
    for (int c = 0; c < kPerBin; ++c) {
      if ((uint32_t)c < at) {
        atomicAdd(&h[ek[c] & (kH3Bins - 1)], 1u);
        const uint32_t slot = atomicAdd(&n2, 1u);
        if (slot < (uint32_t)kC2Cap) {
          c2key[slot] = ek[c];
          c2reg[slot] = (uint16_t)r;
        }
      }
    }
  }
  if (slow) atomicOr(&n2, 0x80000000u);  // members beyond rbin: take all from rband
  __syncthreads();
  if (n2 & 0x80000000u) {
    __syncthreads();  // every thread has read n2
    if (tid == 0) n2 = 0u;
    for (int i = tid; i < kH3Bins; i += NT) h[i] = 0u;
#pragma unroll 1
    for (int r0 = 0; r0 < G; r0 += NT) {
      const int r = r0 + tid;
      uint32_t above = 0u, at = 0u;
      if (r < G) {
        const uint2 cnt = rcnt[r];
        const uint32_t bw = cnt.y & 0x7FFFFFFFu;
        if (bw && !(cnt.y >> 31)) {
          const uint32_t* sr = rsuf + (size_t)r * kH2Bins;
          above = sr[B2];
          at = (B2 ? sr[B2 - 1] : bw) - above;
        }
      }
      uint32_t tot;
      const uint32_t ex = block_scan<NT>(at, wsum, &tot);  // (its barriers order the reset above)
      off[tid] = ex;
      abv[tid] = above;
      __syncthreads();
#pragma unroll 1
      for (uint32_t j = tid; j < tot; j += NT) {
        int a = 0, b = NT - 1;  // the last region slot with off <= j holds member j
        while (a < b) {
          const int m = (a + b + 1) >> 1;
          if (off[m] <= j) a = m; else b = m - 1;
        }
        const uint32_t key = rband[(size_t)(r0 + a) * rcap + abv[a] + (j - off[a])];
        atomicAdd(&h[key & (kH3Bins - 1)], 1u);
        const uint32_t slot = atomicAdd(&n2, 1u);
        if (slot < (uint32_t)kC2Cap) {
          c2key[slot] = key;
          c2reg[slot] = (uint16_t)(r0 + a);
        }
      }
      __syncthreads();
    }
  }
  // class-2 members of the regions without stored band keys: from the lines
  // of those that hold any (their count is known from rsuf)
  const uint32_t thr2 = cls21 << kH2Shift;
  auto in_cls2 = [&](int, uint32_t key) -> bool { return (key >> kH2Shift) == cls21; };
  auto lines_class2 = [&](int wlim, auto f) {
#pragma unroll 1
    for (int wi = 0; wi * 32 < wlim; ++wi) {
      uint32_t m = c2bits[wi];
#pragma unroll 1
      while (m) {
        const int r = wi * 32 + __ffs(m) - 1;
        m &= m - 1u;
        if (r >= wlim) break;
        LineSpan lr;
        lr.load(tiles, summ, nlines, ((int64_t)r * NT + tid) * lpt, lpt);
        walk_mask(lr, lr.flagged([&](int) -> uint32_t { return thr2; }), in_cls2,
                  [&](int, const TileDesc&, int, float, uint32_t key) { f(key); });
      }
    }
  };
  lines_class2(G, [&](uint32_t key) { atomicAdd(&h[key & (kH3Bins - 1)], 1u); });
  __syncthreads();
  block_pick<NT, kH3Bins, 1>(h, need2, wsum, res);
  const uint32_t T = (cls21 << 10) | res[0];
  const uint32_t need3 = (res[1] < need2) ? need2 - res[1] : 0u;

  // class-2 members above T and equal to T in the regions before this one
  uint32_t eqb = 0u;
  auto tally = [&](uint32_t key) {
    gtb += (key > T) ? 1u : 0u;
    eqb += (key == T) ? 1u : 0u;
  };
  if (n2 <= (uint32_t)kC2Cap) {
    for (uint32_t j = tid; j < n2; j += NT)
      if ((int)c2reg[j] < w) tally(c2key[j]);
  } else {
    for_class2<NT>(w, B2, rcap, rcnt, rsuf, rband, off, abv, wsum, tally);
  }
  lines_class2(w, tally);

  // this region: its stored candidate (at most one per thread), or its
  // lines. Counts of (key > T) and (key == T) in position order (the rounds
  // count theirs as they go).
  LineSpan ls;
  uint32_t mask = 0u;
  if (own_ov) {
    ls.load(tiles, summ, nlines, ((int64_t)w * NT + tid) * lpt, lpt);
    mask = ls.flagged([&](int) -> uint32_t { return T; });
  }
  auto at_least_T = [&](int, uint32_t key) -> bool { return key >= T; };
  uint32_t gt = 0u, eq = 0u;
  auto count = [&](float x) {
    const uint32_t key = mag_key(x);
    gt += (key > T) ? 1u : 0u;
    eq += (key == T) ? 1u : 0u;
  };
  if (own_ov) {
    walk_mask(ls, mask, at_least_T,
              [&](int, const TileDesc&, int, float x, uint32_t) { count(x); });
  } else if (cb < ce) {
    count(__uint_as_float(v0.y));  // (fetched at the start)
  }
  const uint32_t sv[4] = {gt, eq, gtb, eqb};
  uint32_t pre[4], tot[4];
  block_scan4<NT>(sv, wsum, pre, tot);
  // clear the part of the zero-initialised scratch that only the earlier
  // kernels of this execution use (not read here), for the next execution
#pragma unroll 1
  for (int64_t i = (int64_t)w * NT + tid; i < clear_words; i += (int64_t)G * NT)
    clear_next[i] = 0u;
  // Other workgroups read the lines of the regions whose band keys were not
  // stored (their level-2 class members, above), so such a region does not
  // zero its residuals here: it records its range of output slots, and the
  // last workgroup to finish zeroes the residuals at those slots' indices.
  const bool defer = (mine.y >> 31) != 0u;
  if (defer && tid == 0) {
    const uint32_t lo = tot[2] + min(tot[3], need3);
    const uint32_t hi = tot[2] + tot[0] + min(tot[3] + tot[1], need3);
    rzr[w] = (uint64_t)min(lo, k) | ((uint64_t)min(hi, k) << 32);
  }
  uint32_t gtr = tot[2] + pre[0];
  uint32_t eqr = tot[3] + pre[1];
  // write
  auto write = [&](uint32_t gidx, float* rp, float x) {
    const uint32_t key = mag_key(x);
    if (key < T) return;
    uint32_t pos = 0xFFFFFFFFu;
    if (key > T) {
      pos = gtr + min(eqr, need3);
      ++gtr;
    } else {
      if (eqr < need3) pos = gtr + eqr;
      ++eqr;
    }
    if (pos < k) {
      idx_out[pos] = (int32_t)gidx;
      put_val(val_out, pos, x, val16);
      if (!defer) *gptr(rp) = 0.0f;
    }
  };
  if (rounds) {
    // elements above T and equal to T before the round (uniform); per
    // round one scan of both counts, packed in 16-bit halves (a round
    // holds at most NT of each)
    uint32_t gtr_r = tot[2], eqr_r = tot[3];
    uint4 cur = v0;
#pragma unroll 1
    for (uint32_t r0 = 0; r0 < mine.x; r0 += NT) {
      const uint32_t j = r0 + (uint32_t)tid;
      const uint4 nxt = mc[min(j + (uint32_t)NT, mine.x - 1u)];  // next round's (clamped)
      const bool have = j < mine.x;
      const float x = __uint_as_float(cur.y);
      const uint32_t key = mag_key(x);
      const bool isg = have && key > T, ise = have && key == T;
      uint32_t rt;
      const uint32_t rp = block_scan<NT>((isg ? 1u : 0u) | (ise ? 0x10000u : 0u), wsum, &rt);
      const uint32_t gbef = gtr_r + (rp & 0xFFFFu), ebef = eqr_r + (rp >> 16);
      uint32_t pos = 0xFFFFFFFFu;
      if (isg) pos = gbef + min(ebef, need3);
      else if (ise && ebef < need3) pos = gbef + ebef;
      if (pos < k) {
        idx_out[pos] = (int32_t)cur.x;
        put_val(val_out, pos, x, val16);
        *gptr(reinterpret_cast<float*>(((uint64_t)cur.w << 32) | cur.z)) = 0.0f;
      }
      gtr_r += rt & 0xFFFFu;
      eqr_r += rt >> 16;
      cur = nxt;
    }
  } else if (gt + eq == 0u) {
    // nothing to write
  } else if (own_ov) {
    walk_mask(ls, mask, at_least_T, [&](int, const TileDesc& t, int e, float x, uint32_t) {
      write((uint32_t)(t.gstart + e), t.r + e, x);
    });
  } else if (cb < ce) {
    write(v0.x, reinterpret_cast<float*>(((uint64_t)v0.w << 32) | v0.z), __uint_as_float(v0.y));
  }
  if (!any_unstored) return;  // (uniform) the common case ends here
  // Every workgroup has read all it reads of the unstored regions' lines and
  // written its outputs; the one that takes the last ticket zeroes the
  // deferred residuals. No workgroup waits for another.
  __syncthreads();
  if (tid == 0) {
    __threadfence();
    last = (atomicAdd(ticket, 1u) == (uint32_t)G - 1u) ? 1u : 0u;
    __threadfence();
  }
  __syncthreads();
  if (!last) return;
  const int32_t ntiles = (int32_t)(nlines / kLinesPerTile);
#pragma unroll 1
  for (int wi = 0; wi * 32 < G; ++wi) {
    uint32_t m = ovbits[wi];
#pragma unroll 1
    while (m) {
      const int r = wi * 32 + __ffs(m) - 1;
      m &= m - 1u;
      const uint64_t rg = __hip_atomic_load(&rzr[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll 1
      for (uint32_t j = (uint32_t)rg + tid; j < (uint32_t)(rg >> 32); j += NT) {
        const int32_t gi = __hip_atomic_load(&idx_out[j], __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        int a = 0, b = ntiles - 1;  // the last tile starting at or before gi
        while (a < b) {
          const int mid = (a + b + 1) >> 1;
          if (tiles[mid].gstart <= gi) a = mid; else b = mid - 1;
        }
        const TileDesc t = tiles[a];
        gptr(t.r)[gi - t.gstart] = 0.0f;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Several selection groups (per-tensor top-k): pick 1, gather, pick 2, hist3,
// pick 3, groupscan, emit. The picks run as k_pick, one workgroup per group.
//
// gather: over the lines whose summary can hold a key of at least the
// group's level-1 bin B1: (a) the level-2 histogram of the elements in bin
// B1 (counted in LDS for the group of the region's first line, which holds
// most of a region's lines when tensors are large, and added to the global
// histogram once; other groups' members go to it directly); (b) ordered
// compaction of all elements with key >= B1 << 20 into `cand`. meta[0] =
// overflow (the candidates did not fit in `cap`; later steps then read
// lines), meta[1] = candidate count.
__global__ __launch_bounds__(kSBlock) void k_gather(const TileDesc* __restrict__ tiles,
                                                    const GroupState* __restrict__ st,
                                                    const uint16_t* __restrict__ summ,
                                                    int64_t nlines, int lpt,
                                                    uint32_t* __restrict__ hist2,
                                                    uint64_t* __restrict__ flags,
                                                    uint2* __restrict__ cand, uint32_t cap,
                                                    uint32_t* __restrict__ meta,
                                                    uint32_t* __restrict__ status) {
  __shared__ uint32_t wsum[2 * kSWaves];
  __shared__ uint64_t red[kSWaves];
  // [slot][thread]: position in the tile (the thread's lines lie in one tile), x
  __shared__ uint16_t stage_e[kGStage * kSBlock];
  __shared__ float stage_x[kGStage * kSBlock];
  __shared__ uint32_t h2[kH2Bins];
  const int tid = threadIdx.x;
  for (int i = tid; i < kH2Bins; i += kSBlock) h2[i] = 0u;
  LineSpan ls;
  const int64_t l0 = (int64_t)blockIdx.x * kSBlock * lpt;  // the region's first line
  ls.load(tiles, summ, nlines, l0 + (int64_t)tid * lpt, lpt);
  const int g0 = l0 < nlines ? tiles[l0 / kLinesPerTile].group : -1;
  __syncthreads();  // h2 cleared
  // B1 = 0xFFFFFFFF for a group with nothing to select: shifted, it lies
  // above every key, so such a group yields no candidates
  const uint32_t b1t = st[ls.t.group].prefix;
  auto b1_of = [&](int) -> uint32_t { return b1t; };
  const uint32_t mask = ls.flagged([&](int g) -> uint32_t { return b1_of(g) << kH1Shift; });
  auto is_cand = [&](int g, uint32_t k) -> bool { return k >= (b1_of(g) << kH1Shift); };
  uint32_t c = 0u;
  walk_mask(ls, mask, is_cand, [&](int, const TileDesc& t, int e, float x, uint32_t k) {
    if (c < (uint32_t)kGStage) {
      stage_e[c * kSBlock + tid] = (uint16_t)e;
      stage_x[c * kSBlock + tid] = x;
    }
    ++c;
    if ((k >> kH1Shift) == b1_of(t.group)) {
      const uint32_t b2 = (k >> kH2Shift) & (kH2Bins - 1);
      if (t.group == g0) atomicAdd(&h2[b2], 1u);
      else atomicAdd(&hist2[(size_t)t.group * kH2Bins + b2], 1u);
    }
  });

  // ordered positions: scan within the workgroup, prefix across workgroups
  // (the scan's barriers also complete the LDS histogram)
  uint32_t total;
  const uint32_t ex = sblock_scan(c, wsum, &total);
  if (g0 >= 0)
    for (int i = tid; i < kH2Bins; i += kSBlock)
      if (h2[i]) atomicAdd(&hist2[(size_t)g0 * kH2Bins + i], h2[i]);
  bool ok;
  const uint64_t pre = group_prefix(flags, total, red, status, &ok);
  // (an incomplete prefix counts as an overflow: the later kernels then
  // read the lines instead of the candidate list)
  const bool fits = ok && pre + total <= cap;
  if (tid == 0) {
    if (!fits) atomicOr(&meta[0], 1u);
    if (blockIdx.x == gridDim.x - 1) meta[1] = (uint32_t)min(pre + total, (uint64_t)0xFFFFFFFFu);
  }
  if (fits && c) {
    const uint64_t pos = pre + ex;
    const uint32_t ns = min(c, (uint32_t)kGStage);
    const uint32_t tcode = (uint32_t)ls.tile << kCandShift;
#pragma unroll 1
    for (uint32_t q = 0; q < ns; ++q)
      cand[pos + q] = make_uint2(tcode | stage_e[q * kSBlock + tid],
                                 __float_as_uint(stage_x[q * kSBlock + tid]));
    if (c > (uint32_t)kGStage) {  // rare: read the lines again for the rest
      uint32_t i = 0u;
      walk_mask(ls, mask, is_cand, [&](int tile, const TileDesc&, int e, float x, uint32_t) {
        if (i >= (uint32_t)kGStage)
          cand[pos + i] = make_uint2(((uint32_t)tile << kCandShift) | (uint32_t)e, __float_as_uint(x));
        ++i;
      });
    }
  }
}

// hist3: per-group histogram of the low 10 key bits over the group's level-2
// class (key >> 10 == its 21-bit prefix), read from the candidates (or the
// lines after an overflow).
__global__ __launch_bounds__(kSBlock) void k_hist3(const TileDesc* __restrict__ tiles,
                                                   int32_t ntiles,
                                                   const GroupState* __restrict__ st,
                                                   const uint16_t* __restrict__ summ,
                                                   int64_t nlines, int lpt,
                                                   const uint2* __restrict__ cand,
                                                   const uint32_t* __restrict__ meta,
                                                   uint32_t* __restrict__ hist3) {
  const int tid = threadIdx.x;
  const uint32_t ov = meta[0], C = meta[1];
  auto cls_of = [&](int g) -> uint32_t {
    const GroupState sg = st[g];
    return sg.need ? sg.prefix : 0xFFFFFFFFu;
  };
  auto in_cls = [&](int g, uint32_t k) -> bool { return (k >> kH2Shift) == cls_of(g); };
  auto body = [&](int, const TileDesc& t, int, float, uint32_t k) {
    if (in_cls(t.group, k)) atomicAdd(&hist3[(size_t)t.group * kH3Bins + (k & (kH3Bins - 1))], 1u);
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
    for (uint32_t j = wb + 4 * tid; j < we; j += 4 * kSBlock)
      walk_cands(tiles, ntiles, cand, j, min(j + 4u, we), body);
  }
}

// groupscan: base[2g] = sum over earlier groups of #{key > T}, base[2g + 1] =
// the same for #{key == T} (counting only the equal keys that are kept).
__global__ __launch_bounds__(kSBlock) void k_groupscan(const GroupDesc* __restrict__ groups,
                                                       const GroupState* __restrict__ st,
                                                       int32_t ngroups,
                                                       uint32_t* __restrict__ base) {
  __shared__ uint32_t wsum[2 * kSWaves];
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
    uint2 t;
    const uint2 x = block_scan2<kSBlock>(gt, eq, wsum, &t);
    if (g < ngroups) {
      base[2 * g] = carry_gt + x.x;
      base[2 * g + 1] = carry_eq + x.y;
    }
    carry_gt += t.x;
    carry_eq += t.y;
  }
}

// emit: ordered compaction of the selection. An element of group g with
// key > T_g goes to slot (#gt before it in g) + min(#eq before it in g,
// need_g); an element with key == T_g is kept while fewer than need_g equal
// keys precede it in g. Counts before an element are global prefixes (over
// the candidate list, in position order) minus the group's base.
template <bool kFold>
__global__ __launch_bounds__(kSBlock) void k_emit(const TileDesc* __restrict__ tiles,
                                                  int32_t ntiles,
                                                  const GroupDesc* __restrict__ groups,
                                                  const GroupState* __restrict__ st,
                                                  const uint16_t* __restrict__ summ,
                                                  int64_t nlines, int lpt,
                                                  const uint2* __restrict__ cand,
                                                  const uint32_t* __restrict__ meta,
                                                  const uint32_t* __restrict__ base,
                                                  uint64_t* __restrict__ flags,
                                                  int32_t* __restrict__ idx_out,
                                                  void* __restrict__ val_out, int val16,
                                                  uint32_t* __restrict__ status,
                                                  uint32_t* __restrict__ clear_next,
                                                  int64_t clear_words, int32_t fold_ngroups) {
  __shared__ uint32_t wsum[2 * kSWaves];
  __shared__ uint64_t red[kSWaves];
  __shared__ int32_t stage_code[kStage * kSBlock];  // [slot][thread]: (tile << 13) | e
  __shared__ float stage_x[kStage * kSBlock];
  __shared__ uint2 lbase[kEmitLdsGroups];
  __shared__ uint4 lgrp[kEmitLdsGroups];  // per group: T, need, k, out_base
  const int tid = threadIdx.x;
  // With kFold (fold_ngroups, at most kEmitLdsGroups, groups) every workgroup
  // forms the groups' bases itself (what k_groupscan writes into base[]):
  // the groups' results are fetched now and scanned after pass 1, and what
  // the writes need of each group is kept in LDS.
  uint32_t fgt = 0u, feq = 0u;
  if (tid < fold_ngroups) {
    const GroupState sg = st[tid];
    const GroupDesc gd = groups[tid];
    fgt = (gd.k > sg.need) ? gd.k - sg.need : 0u;
    feq = sg.need ? sg.n_eq : 0u;
    lgrp[tid] = make_uint4(sg.T, sg.need, gd.k, gd.out_base);
  }
  if constexpr (kFold) __syncthreads();
  // clear the part of the zero-initialised scratch that only the earlier
  // kernels of this execution use (not read here), for the next execution
#pragma unroll 1
  for (int64_t i = (int64_t)blockIdx.x * kSBlock + tid; i < clear_words;
       i += (int64_t)gridDim.x * kSBlock)
    clear_next[i] = 0u;
  const uint32_t ov = meta[0], C = meta[1];
  auto T_of = [&](int g) -> uint32_t {
    if constexpr (kFold) return lgrp[g].x;
    else return st[g].T;
  };
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
  if constexpr (kFold) {  // (its barriers also order lbase for the writes)
    uint2 gtot;
    const uint2 gx = block_scan2<kSBlock>(fgt, feq, wsum, &gtot);
    if (tid < fold_ngroups) lbase[tid] = gx;
  }
  uint2 tot;
  const uint2 x2 = block_scan2<kSBlock>(gt, eq, wsum, &tot);
  bool ok;
  const uint64_t pre =
      group_prefix(flags, (uint64_t)tot.x | ((uint64_t)tot.y << 31), red, status, &ok);
  if (nst == 0u || !ok) return;  // (no place is known without the full prefix)
  uint32_t gtr = (uint32_t)(pre & 0x7FFFFFFFu) + x2.x;
  uint32_t eqr = (uint32_t)((pre >> 31) & 0x7FFFFFFFu) + x2.y;
  // pass 2: write
  auto write = [&](int, const TileDesc& t, int e, float x, uint32_t k) {
    const int g = t.group;
    uint32_t T, need, gk, gob, bg, be;
    if constexpr (kFold) {
      const uint4 q = lgrp[g];
      T = q.x;
      need = q.y;
      gk = q.z;
      gob = q.w;
      bg = lbase[g].x;
      be = lbase[g].y;
    } else {
      const GroupState sg = st[g];
      const GroupDesc gd = groups[g];
      T = sg.T;
      need = sg.need;
      gk = gd.k;
      gob = gd.out_base;
      bg = base[2 * g];
      be = base[2 * g + 1];
    }
    if (k < T) return;
    uint32_t pos = 0xFFFFFFFFu;
    if (k > T) {
      pos = (gtr - bg) + min(eqr - be, need);
      ++gtr;
    } else {
      if (eqr - be < need) pos = (gtr - bg) + (eqr - be);
      ++eqr;
    }
    if (pos < gk) {
      idx_out[gob + pos] = t.gstart + e;
      put_val(val_out, (size_t)gob + pos, x, val16);
      gptr(t.r)[e] = 0.0f;
    }
  };
  if (nst <= (uint32_t)kStage) {
    // the staged elements' tile descriptors are all requested before the
    // first write
    TileDesc td[kStage];
#pragma unroll
    for (int q = 0; q < kStage; ++q)
      if ((uint32_t)q < nst) td[q] = tiles[(uint32_t)stage_code[q * kSBlock + tid] >> kCandShift];
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
      if ((uint32_t)q < nst) {
        const uint32_t code = (uint32_t)stage_code[q * kSBlock + tid];
        const float x = stage_x[q * kSBlock + tid];
        write((int)(code >> kCandShift), td[q], (int)(code & (kTile - 1)), x, mag_key(x));
      }
    }
  } else if (ov) {
    walk_mask(ls, mask, at_least_T, write);
  } else {
    walk_cands(tiles, ntiles, cand, cb, ce, write);
  }
}

// ---------------------------------------------------------------------------
// The P workers' lists, in one of two forms: the gathered layout (worker p's
// entries at p * stride, nnz[p] of them, or stride without nnz) or a table of
// per-worker pointers and counts (kTable).
struct ListsArg {
  const int32_t* idx;        // gathered form
  const void* val;
  int64_t stride;
  const int32_t* nnz;
  const WorkerList* table;   // per-worker form
};
typedef __attribute__((address_space(1))) const int32_t gint;

// seg: seg[u * P + p] = first entry of worker p's list whose index lies in
// update tile u or later; seg[ntiles_u * P + p] = nnz_p. Tile-major, so the
// workgroup of tile u reads two contiguous rows. Also flags unsorted or
// out-of-range lists in the status word.
template <bool kTable>
__global__ void k_seg(ListsArg lists, int32_t P, int32_t d, int32_t ntiles_u,
                      int32_t* __restrict__ seg, uint32_t* __restrict__ status) {
  const int p = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int32_t i_here = 0, i_prev = 0;
  int64_t n;
  if constexpr (kTable) {
    const WorkerList wl = lists.table[p];
    n = wl.n;
    if (j < n) {
      const gint* L = (const gint*)wl.idx;
      i_here = L[j];
      i_prev = L[j > 0 ? j - 1 : 0];
    }
  } else {
    // this entry and the one before it, read before the count is known
    // (every j < stride is inside the list's storage), so all three loads
    // overlap; no storage at all for stride == 0 (a kernel-wide value)
    const int64_t stride = lists.stride;
    const int32_t* __restrict__ L = lists.idx + (int64_t)p * stride;
    const int64_t jc = j < stride ? j : stride - 1;
    if (stride > 0) {
      i_here = L[jc];
      i_prev = L[jc > 0 ? jc - 1 : 0];
    }
    n = lists.nnz ? (int64_t)lists.nnz[p] : stride;
    n = n < 0 ? 0 : (n > stride ? stride : n);
  }
  if (n == 0) {
    for (int64_t u = j; u <= ntiles_u; u += (int64_t)gridDim.x * blockDim.x)
      seg[u * P + p] = 0;
    return;
  }
  if (j >= n) return;
  auto tile_of = [&](int32_t i) -> int32_t {
    return i < 0 ? 0 : (i >= d ? ntiles_u - 1 : (i >> kUShift));
  };
  const int32_t i = i_here;
  uint32_t bad = (i < 0 || i >= d) ? TKEF_STATUS_INDEX_RANGE : 0u;
  const int32_t t = tile_of(i);
  int32_t tp = -1;
  if (j > 0) {
    const int32_t ip = i_prev;
    if (ip > i) bad |= TKEF_STATUS_UNSORTED;
    tp = tile_of(ip);
  }
  for (int32_t u = tp + 1; u <= t; ++u) seg[(int64_t)u * P + p] = (int32_t)j;
  if (j == n - 1)
    for (int32_t u = t + 1; u <= ntiles_u; ++u) seg[(int64_t)u * P + p] = (int32_t)n;
  if (bad && status) atomicOr(status, bad);
}

// ---------------------------------------------------------------------------
// update: one workgroup per update tile. op: kOpSgd (every position: weight
// decay and optional momentum), kOpSparseSgd (mu = wd = 0: only the positions
// some list names), kOpAggregate (no step: the tile's sums G are written into
// the bound tensors, every position, zero where no list names it).
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

// LARS step (the cited method's update with the rate of Eq. lars):
// D = G + eps w; U = rate D; b = mu b + U and w - b (momentum), else w - U.
__device__ __forceinline__ float lars_step(float G, float w, float& b, bool mom, float rate,
                                           float mu, float eps) {
  const float decay = eps * w;
  const float D = G + decay;
  const float U = rate * D;
  if (mom) {
    const float keep = mu * b;
    b = keep + U;
    return w - b;
  }
  return w - U;
}

// Sum of two doubles per thread over a kUBlock-thread workgroup, in a fixed
// order (wave butterflies, then the waves in order). red: 2 * kUBlock / 64
// doubles of LDS. Result valid in thread 0; ends with a barrier.
__device__ __forceinline__ double2 ublock_sum2(double a, double b, double* red) {
  constexpr int NW = kUBlock / 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  if ((tid & 63) == 0) {
    red[tid >> 6] = a;
    red[NW + (tid >> 6)] = b;
  }
  __syncthreads();
  double2 r = make_double2(0.0, 0.0);
  if (tid == 0) {
    for (int i = 0; i < NW; ++i) {
      r.x += red[i];
      r.y += red[NW + i];
    }
  }
  __syncthreads();
  return r;
}

constexpr int kXcds = 8;                      // MI355X: 8 accelerator dies
constexpr int kXcdRun = 16;                   // consecutive update tiles one die takes
constexpr int kUVecPerThread = kUTile / 4 / kUBlock;  // float4 per thread per tile

constexpr int kPairUnroll = 4;  // list entries per thread and chunk of the accumulation
constexpr int kUOwn = kUTile / kUBlock;  // tile positions one thread owns in the ordered sum

// The ordered accumulation of one chunk of list entries (deterministic mode).
// Entry j * kUBlock + tid of the chunk (li[j], vv[j]; li outside [0, len)
// for none) is the chunk's entry number j * kUBlock + tid, and the entries
// are numbered in worker order, then list order, as Alg. 2 visits them.
// Each position's entries are added to acc in that order, one binary32 add
// at a time, so the sums do not depend on the order in which threads run:
//   1. LDS counters count every position's entries (word w holds the 16-bit
//      counts of positions w and w + kUTile / 2); each entry keeps its
//      arrival rank at its position;
//   2. thread t owns the words t, t + kUBlock, ... (so a wavefront's LDS
//      accesses fall in distinct banks) and with them kUOwn positions: an
//      exclusive scan of the counts gives every position a first slot (the
//      positions' slot ranges are disjoint; their order does not matter);
//   3. each entry goes to slot first + rank of (dq: entry number, dv: value);
//   4. each owner sorts its positions' slots by entry number (insertion
//      sort; a position usually has one entry) and adds them in that order.
// dcnt: kUTile / 2 words, zero on entry and on return; dq, dv: kUBlock *
// kPairUnroll slots; dws: kUBlock / 64 words. Uniform in the workgroup.
__device__ __forceinline__ void det_accumulate(const int32_t (&li)[kPairUnroll],
                                               const float (&vv)[kPairUnroll], int32_t len,
                                               bool sparse_mode, float* acc, uint32_t* mask,
                                               uint32_t* dcnt, uint16_t* dq, float* dv,
                                               uint32_t* dws) {
  static_assert(kUBlock * kPairUnroll <= 65535, "slots and entry numbers fit 16 bits");
  static_assert(kUOwn % 2 == 0, "two counts per word");
  constexpr int kHalf = kUTile / 2;  // position p: word p % kHalf, half p / kHalf
  constexpr int kWords = kUOwn / 2;  // words per thread
  const int tid = threadIdx.x;
  uint32_t rank[kPairUnroll];
#pragma unroll
  for (int j = 0; j < kPairUnroll; ++j) {
    rank[j] = 0u;
    if (li[j] >= 0 && li[j] < len) {
      const uint32_t sh = li[j] >= kHalf ? 16u : 0u;
      rank[j] = (atomicAdd(&dcnt[li[j] & (kHalf - 1)], 1u << sh) >> sh) & 0xFFFFu;
    }
  }
  __syncthreads();
  uint32_t cw[kWords];  // this thread's counts, two per word
  uint32_t mine = 0u;
#pragma unroll
  for (int i = 0; i < kWords; ++i) {
    cw[i] = dcnt[tid + i * kUBlock];
    mine += (cw[i] & 0xFFFFu) + (cw[i] >> 16);
  }
  uint32_t total;
  const uint32_t first = block_scan<kUBlock>(mine, dws, &total);  // (ends with a barrier)
  uint32_t o = first;
#pragma unroll
  for (int i = 0; i < kWords; ++i) {
    const uint32_t c0 = cw[i] & 0xFFFFu, c1 = cw[i] >> 16;
    dcnt[tid + i * kUBlock] = o | ((o + c0) << 16);  // first slots
    o += c0 + c1;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPairUnroll; ++j) {
    if (li[j] >= 0 && li[j] < len) {
      const uint32_t sh = li[j] >= kHalf ? 16u : 0u;
      const uint32_t slot = ((dcnt[li[j] & (kHalf - 1)] >> sh) & 0xFFFFu) + rank[j];
      dq[slot] = (uint16_t)(j * kUBlock + tid);
      dv[slot] = vv[j];
    }
  }
  __syncthreads();
  o = first;
#pragma unroll 1
  for (int i = 0; i < kUOwn; ++i) {
    const uint32_t c = (i & 1) ? (cw[i >> 1] >> 16) : (cw[i >> 1] & 0xFFFFu);
    if (c == 0u) continue;
    const uint32_t e = o + c;
#pragma unroll 1
    for (uint32_t a = o + 1; a < e; ++a) {
      const uint16_t kq = dq[a];
      const float kv = dv[a];
      uint32_t b = a;
      while (b > o && dq[b - 1] > kq) {
        dq[b] = dq[b - 1];
        dv[b] = dv[b - 1];
        --b;
      }
      dq[b] = kq;
      dv[b] = kv;
    }
    const int pos = tid + (i >> 1) * kUBlock + (i & 1) * kHalf;
    float sum = acc[pos];
#pragma unroll 1
    for (uint32_t a = o; a < e; ++a) sum = sum + dv[a];
    acc[pos] = sum;
    if (sparse_mode) atomicOr(&mask[pos >> 5], 1u << (pos & 31));
    o = e;
  }
#pragma unroll
  for (int i = 0; i < kWords; ++i) dcnt[tid + i * kUBlock] = 0u;
  __syncthreads();
}

// kLars: the LARS norm and step passes (a separate instantiation, so the SGD
// and aggregation passes keep their register budget).
// kTable: the lists come as a table of per-worker pointers (binary32 values).
// kDet: each position's entries are added in worker order (det_accumulate)
// instead of by LDS float atomics in any order.
template <bool kLars, bool kTable, bool kDet>
__global__ __launch_bounds__(kUBlock) void k_update(
    const UpdTensor* __restrict__ tens, const int32_t* __restrict__ tile_first, int32_t ntens,
    int32_t d, int32_t ntiles_u, ListsArg lists, int val16, int32_t P,
    const int32_t* __restrict__ seg, float lr, float mu, float wd, int op, int has_mom,
    LarsArgs lars) {
  static_assert(!(kLars && kTable), "LARS takes the gathered lists");
  const int32_t* __restrict__ idx = lists.idx;
  const void* __restrict__ val = lists.val;
  const int64_t stride = lists.stride;
  const int32_t* __restrict__ nnz = lists.nnz;
  const bool sparse_mode = op == kOpSparseSgd;
  const bool densify = op == kOpAggregate;
  const bool lnorm = kLars && op == kOpLarsNorm;
  const bool lapply = kLars && op == kOpLarsApply;
  __shared__ double lred[2 * kUBlock / 64];
  __shared__ __align__(16) float acc[kUTile];
  __shared__ uint32_t mask[kUTile / 32];
  __shared__ int32_t sbeg[kUBlock];
  __shared__ uint32_t scan[kUBlock];
  // per-worker form: the list pointers of the current batch of workers
  __shared__ const int32_t* s_ip[kTable ? kUBlock : 1];
  __shared__ const float* s_vp[kTable ? kUBlock : 1];
  // deterministic mode: counters, slots and scan words of det_accumulate
  __shared__ uint32_t dcnt[kDet ? kUTile / 2 : 1];
  __shared__ uint16_t dq[kDet ? kUBlock * kPairUnroll : 1];
  __shared__ float dv[kDet ? kUBlock * kPairUnroll : 1];
  __shared__ uint32_t dws[kDet ? kUBlock / 64 : 1];
  const int tid = threadIdx.x;
  // Workgroups go round-robin to the XCDs; give each XCD runs of kXcdRun
  // consecutive tiles, so that neighbouring tiles, which share the cache
  // lines at the ends of every worker's list segment, are mostly served by
  // one L2, while the dies still stream from nearby addresses (one run of
  // the whole range per die streamed 6 us slower; runs of 4 / 8 / 16 / 32 /
  // 128 tiles: 79.6 / 77.8 / 77.5 / 78.8 / 82.4 us against 82.3).
  const int q = (int)(blockIdx.x / kXcds);
  const int u = (q / kXcdRun) * (kXcds * kXcdRun) + (int)(blockIdx.x % kXcds) * kXcdRun +
                q % kXcdRun;
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
  if (fast && !densify) {  // (aggregation only writes the tile)
    const float4* w4 = reinterpret_cast<const float4*>(w_tile);
    const float4* b4 = reinterpret_cast<const float4*>(b_tile);
#pragma unroll
    for (int q = 0; q < kUVecPerThread; ++q) {
      // (the norm pass reads w again in the step pass: keep it cached)
      wv[q] = lnorm ? w4[q * kUBlock + tid] : load_nt4(w4 + q * kUBlock + tid);
      if (mom && !lnorm) bv[q] = load_nt4(b4 + q * kUBlock + tid);
    }
  }

  for (int i = tid; i < kUTile; i += kUBlock) acc[i] = 0.0f;
  if (sparse_mode)
    for (int i = tid; i < kUTile / 32; i += kUBlock) mask[i] = 0u;
  if constexpr (kDet)
    for (int i = tid; i < kUTile / 2; i += kUBlock) dcnt[i] = 0u;
  __syncthreads();

  // 1. accumulate every worker's entries that fall in this tile
  for (int p0 = 0; p0 < P; p0 += kUBlock) {
    const int p = p0 + tid;
    int32_t b = 0, e = 0;
    if (p < P) {
      int64_t np;
      if constexpr (kTable) {
        const WorkerList wl = lists.table[p];
        np = wl.n;
        s_ip[tid] = wl.idx;
        s_vp[tid] = static_cast<const float*>(wl.val);
      } else {
        np = nnz ? (int64_t)nnz[p] : stride;
        np = np < 0 ? 0 : (np > stride ? stride : np);
      }
      int64_t sb = seg[(int64_t)u * P + p], se = seg[(int64_t)(u + 1) * P + p];
      sb = sb < 0 ? 0 : (sb > np ? np : sb);
      se = se < sb ? sb : (se > np ? np : se);
      b = (int32_t)sb;
      e = (int32_t)se;
    }
    sbeg[tid] = b;
    // inclusive prefix of the segment lengths, for the entry -> worker search
    // (block_scan ends with a barrier, so scan[] can be rewritten here)
    uint32_t total;
    const uint32_t ex = block_scan<kUBlock>((uint32_t)(e - b), scan, &total);
    scan[tid] = ex + (uint32_t)(e - b);
    __syncthreads();
    // entries of this batch of workers, kPairUnroll per thread with all
    // their loads in flight before the LDS adds
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
          const int64_t jj = (int64_t)sbeg[lo] + (q - before);
          if constexpr (kTable) {
            li[j] = ((const gint*)s_ip[lo])[jj] - base;
            vv[j] = ((const gfloat*)s_vp[lo])[jj];
          } else {
            const int64_t gi = (int64_t)(p0 + lo) * stride + jj;
            li[j] = idx[gi] - base;
            vv[j] = get_val(val, (size_t)gi, val16);
          }
        }
      }
      if constexpr (kDet) {
        det_accumulate(li, vv, len, sparse_mode, acc, mask, dcnt, dq, dv, dws);
      } else {
#pragma unroll
        for (int j = 0; j < kPairUnroll; ++j) {
          if (li[j] >= 0 && li[j] < len) {
            atomicAdd(&acc[li[j]], vv[j]);
            if (sparse_mode) atomicOr(&mask[li[j] >> 5], 1u << (li[j] & 31));
          }
        }
      }
    }
    __syncthreads();
  }

  // 2a. LARS norms: per tensor of the tile, sum w^2 and G^2 (double) into
  // its pair
  if (lnorm) {
    const int32_t tl = fast ? t0 : min(tile_first[u + 1], ntens - 1);
    for (int ti = t0; ti <= tl; ++ti) {
      const UpdTensor tt = tens[ti];
      const int64_t a = max((int64_t)base, tt.goff);
      const int64_t z = min((int64_t)base + len, tt.goff + tt.n);
      if (z <= a) continue;  // (uniform in the workgroup)
      double sw = 0.0, sg = 0.0;
      if (fast) {
        const float4* a4 = reinterpret_cast<const float4*>(acc);
#pragma unroll
        for (int q = 0; q < kUVecPerThread; ++q) {
          const float4 G = a4[q * kUBlock + tid];
          const float4 w = wv[q];
          sw += (double)w.x * w.x + (double)w.y * w.y + (double)w.z * w.z + (double)w.w * w.w;
          sg += (double)G.x * G.x + (double)G.y * G.y + (double)G.z * G.z + (double)G.w * G.w;
        }
      } else {
        const gfloat* w = gptr(tt.w + (a - tt.goff));
        const int la = (int)(a - base), cnt = (int)(z - a);
        for (int q = tid; q < cnt; q += kUBlock) {
          const double wq = w[q], gq = acc[la + q];
          sw += wq * wq;
          sg += gq * gq;
        }
      }
      const double2 r = ublock_sum2(sw, sg, lred);
      if (tid == 0) lars.part[lars.tpair[ti] + (u - (int32_t)(tt.goff >> kUShift))] = r;
    }
    return;
  }

  // 2. apply the SGD (or LARS) step
  if (fast) {
    float4* w4 = reinterpret_cast<float4*>(w_tile);
    float4* b4 = reinterpret_cast<float4*>(b_tile);
    const float4* a4 = reinterpret_cast<const float4*>(acc);
#pragma unroll
    for (int q = 0; q < kUVecPerThread; ++q) {
      const int v = q * kUBlock + tid;
      const float4 G = a4[v];
      if (densify) {
        store_nt4(w4 + v, G);
        continue;
      }
      float4 w = wv[q], bb = mom ? bv[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      if (lapply) {
        const float rate = (float)lars.rate[t0];
        w.x = lars_step(G.x, w.x, bb.x, mom, rate, mu, lars.eps);
        w.y = lars_step(G.y, w.y, bb.y, mom, rate, mu, lars.eps);
        w.z = lars_step(G.z, w.z, bb.z, mom, rate, mu, lars.eps);
        w.w = lars_step(G.w, w.w, bb.w, mom, rate, mu, lars.eps);
      } else {
        w.x = sgd_step(G.x, w.x, bb.x, mom, lr, mu, wd);
        w.y = sgd_step(G.y, w.y, bb.y, mom, lr, mu, wd);
        w.z = sgd_step(G.z, w.z, bb.z, mom, lr, mu, wd);
        w.w = sgd_step(G.w, w.w, bb.w, mom, lr, mu, wd);
      }
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
        gfloat* wp = gptr(tens[lo].w + (gi - tens[lo].goff));
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
    gfloat* __restrict__ w = gptr(tt.w + (a - tt.goff));
    gfloat* __restrict__ bm = mom ? gptr(tt.b + (a - tt.goff)) : nullptr;
    const bool vec = ((reinterpret_cast<uintptr_t>(w) |
                       (bm ? reinterpret_cast<uintptr_t>(bm) : 0u)) & 15u) == 0;
    const float rate = lapply ? (float)lars.rate[ti] : 0.0f;
    auto step = [&](float G, float wq, float& bq) -> float {
      return lapply ? lars_step(G, wq, bq, mom, rate, mu, lars.eps)
                    : sgd_step(G, wq, bq, mom, lr, mu, wd);
    };
    int done = 0;
    if (vec) {
      const int nv = cnt >> 2;
      gv4f* w4 = (gv4f*)w;
      gv4f* b4 = (gv4f*)bm;
      for (int q = tid; q < nv; q += kUBlock) {
        if (densify) {
          const int l = la + 4 * q;
          w4[q] = v4f{acc[l], acc[l + 1], acc[l + 2], acc[l + 3]};
          continue;
        }
        const v4f wv4 = w4[q];
        const v4f bv4 = bm ? b4[q] : v4f{0.f, 0.f, 0.f, 0.f};
        float wq[4] = {wv4.x, wv4.y, wv4.z, wv4.w}, bq[4] = {bv4.x, bv4.y, bv4.z, bv4.w};
        const int l = la + 4 * q;
#pragma unroll
        for (int c = 0; c < 4; ++c) wq[c] = step(acc[l + c], wq[c], bq[c]);
        w4[q] = v4f{wq[0], wq[1], wq[2], wq[3]};
        if (mom) b4[q] = v4f{bq[0], bq[1], bq[2], bq[3]};
      }
      done = nv << 2;
    }
    for (int q = done + tid; q < cnt; q += kUBlock) {
      if (densify) {
        w[q] = acc[la + q];
        continue;
      }
      float bq = mom ? bm[q] : 0.0f;
      w[q] = step(acc[la + q], w[q], bq);
      if (mom) bm[q] = bq;
    }
  }
}

// ---------------------------------------------------------------------------
// LARS rates from dense gradients (the layer-wise rates of Eq. lars computed
// for a list of layers): per update tile and tensor, the sums of w^2 and g^2.
__global__ __launch_bounds__(kUBlock) void k_lars_norm_dense(
    const UpdTensor* __restrict__ tens, const float* const* __restrict__ gptrs,
    const int32_t* __restrict__ tile_first, int32_t ntens, int32_t d, int32_t ntiles_u,
    double2* __restrict__ part, const int32_t* __restrict__ tpair) {
  __shared__ double lred[2 * kUBlock / 64];
  const int tid = threadIdx.x;
  const int u = (int)blockIdx.x;  // (no pair lists to share: tiles in address order)
  if (u >= ntiles_u) return;
  const int32_t base = u << kUShift;
  const int32_t len = min(kUTile, d - base);
  const int32_t t0 = tile_first[u], tl = min(tile_first[u + 1], ntens - 1);
  for (int ti = t0; ti <= tl; ++ti) {
    const UpdTensor tt = tens[ti];
    const int64_t a = max((int64_t)base, tt.goff);
    const int64_t z = min((int64_t)base + len, tt.goff + tt.n);
    if (z <= a) continue;
    const gfloat* w = gptr(tt.w + (a - tt.goff));
    const gfloat* g = gptr(gptrs[ti] + (a - tt.goff));
    const int cnt = (int)(z - a);
    double sw = 0.0, sg = 0.0;
    const bool vec = ((reinterpret_cast<uintptr_t>(w) | reinterpret_cast<uintptr_t>(g)) & 15u) == 0;
    int done = 0;
    if (vec) {
      const int nv = cnt >> 2;
      const gv4f* w4 = (const gv4f*)w;
      const gv4f* g4 = (const gv4f*)g;
      for (int q = tid; q < nv; q += kUBlock) {
        const v4f x = __builtin_nontemporal_load(w4 + q);
        const v4f y = __builtin_nontemporal_load(g4 + q);
        sw += (double)x.x * x.x + (double)x.y * x.y + (double)x.z * x.z + (double)x.w * x.w;
        sg += (double)y.x * y.x + (double)y.y * y.y + (double)y.z * y.z + (double)y.w * y.w;
      }
      done = nv << 2;
    }
    for (int q = done + tid; q < cnt; q += kUBlock) {
      const double x = w[q], y = g[q];
      sw += x * x;
      sg += y * y;
    }
    const double2 r = ublock_sum2(sw, sg, lred);
    if (tid == 0) part[tpair[ti] + (u - (int32_t)(tt.goff >> kUShift))] = r;
  }
}

// One workgroup per tensor: its pairs summed in a fixed order, the norms,
// and the rate gamma eta ||w|| / (||g|| + eps ||w||) of Eq. lars wherever the
// denominator is positive (0 for a zero weight norm, gamma eta / eps for a
// zero gradient norm). With eps >= 0 the denominator is zero only when g = 0
// and eps w = 0 on the whole layer; the rate is 0 there (every finite rate
// gives the same step, since D = g + eps w = 0).
__global__ __launch_bounds__(kUBlock) void k_lars_rates(const int32_t* __restrict__ tpair,
                                                        const double2* __restrict__ part,
                                                        double gamma, double eta, double eps,
                                                        double* __restrict__ rate,
                                                        double* __restrict__ rate_out) {
  __shared__ double lred[2 * kUBlock / 64];
  const int t = blockIdx.x, tid = threadIdx.x;
  const int32_t pb = tpair[t], pe = tpair[t + 1];
  double sw = 0.0, sg = 0.0;
  for (int32_t i = pb + tid; i < pe; i += kUBlock) {
    const double2 v = part[i];
    sw += v.x;
    sg += v.y;
  }
  const double2 r = ublock_sum2(sw, sg, lred);
  if (tid == 0) {
    const double nw = sqrt(r.x), ng = sqrt(r.y);
    const double den = ng + eps * nw;
    const double lam = den > 0.0 ? (gamma * eta * nw) / den : 0.0;
    rate[t] = lam;
    if (rate_out) rate_out[t] = lam;
  }
}

// ---------------------------------------------------------------------------
// MSTopK (Alg. 1): the approximate selector. a = |x|; the mean and the
// maximum of a give the trial thresholds mean + ratio * (u - mean); N rounds
// bisect ratio on the count of elements at or above the threshold; the
// result is every element at or above thres1 (the largest count <= k seen)
// plus a run of k - k1 elements, in position order, of the band
// thres2 <= a < thres1 starting at an offset drawn by the caller.
//
// GPU form. Thresholds are compared as magnitude keys: a >= t (a binary32
// widened exactly, t a double) holds exactly when key(a) >= K(t), K(t) the
// key of the smallest binary32 >= t. Bisection is a binary tree, so one pass
// that counts the elements at or above each of the 2^m - 1 thresholds of the
// next m rounds lets the rounds be replayed afterwards exactly as the loop
// would run them. The first pass, over every element, takes m = 6; the later
// ones, over the few lines that reach the bracket, take m = 12: N rounds take
// 1 + ceil((N - 6) / 12) passes (three for N = 30).
//   ms_stream  x = g + r into r, line summaries, the exact sum of |x| (per
//              exponent sums of significands in LDS, then ten 32-bit digits
//              per workgroup added into one of 16 copies) and the largest key
//   ms_count   forms the mean (the exact sum rounded once to double, divided
//              by d) and u, then counts every element against the 63 keys of
//              rounds 1..6
//   ms_refine  replays the previous pass's rounds from its counts, then
//              counts against the next 4095 keys over the lines whose summary
//              can reach the lowest of them (later rounds only look at the
//              top of the distribution)
//   ms_emit    replays the last pass's rounds, fixes K1 = K(thres1),
//              K2 = K(thres2), the window offset and length, and writes the
//              ordered compaction of {key >= K1} and of the window of the
//              band {K2 <= key < K1}; the selected residuals are set to +0
// The small state between passes (mean, u, bracket, recorded counts and
// keys) is recomputed by every workgroup of the next kernel from the totals
// of the previous pass (identical double operations everywhere);
// workgroup 0 also stores it, for the kernels after and for the caller.
// No workgroup waits for another, and no kernel needs a device-wide fence.
namespace {

constexpr int kMsKeys = 64;                // first pass: keys[1..63] (keys[0] unused)
constexpr int kMsRefineKeys = kMsRefineBins;  // later passes: keys[1..4095]
constexpr uint32_t kMsNone = 0x80000000u;  // "no thres1": above every key

// Key of the smallest binary32 >= t, for t >= 0 (0 for t <= 0 or NaN).
__device__ __forceinline__ uint32_t ms_key_ceil(double t) {
  if (!(t > 0.0)) return 0u;
  if (t > 3.4028234663852886e38) return 0x7F800000u;
  const float f = (float)t;  // round to nearest
  uint32_t b = __float_as_uint(f);
  if ((double)f < t) b += 1u;
  return b;
}

// The exact sum of binary32 magnitudes is kept as kMsDigits 32-bit digits
// (units of 2^-149, each digit accumulated in 64 bits so that carries can
// wait): es[E] = the sum of the significands (hidden bit included) of the
// magnitudes with exponent field E contributes es[E] * 2^(max(E, 1) - 1).
// ms_digits_add adds one such term as three digits (es < 2^55 and a shift
// < 254 fit in the 320 bits).
constexpr int kMsDigits = 10;
static_assert(kMsDigits <= kMsDigitStride, "digits per copy");
__device__ __forceinline__ void ms_digits_add(int E, unsigned long long m,
                                              unsigned long long* dig) {
  if (!m) return;
  const int sft = (E ? E : 1) - 1;
  const int q = sft >> 5, o = sft & 31;
  // m << o spans 87 bits at most: three digits from q
  const unsigned long long lo = m << o;                      // bits 0..63 of m << o
  const unsigned long long hi = o ? (m >> (64 - o)) : 0ull;  // bits 64..
  atomicAdd(&dig[q], lo & 0xFFFFFFFFull);
  atomicAdd(&dig[q + 1], lo >> 32);
  if (hi) atomicAdd(&dig[q + 2], hi);
}

// The digits' value rounded once to double (nearest, ties to even). Called
// by one thread; every dig[i] < 2^63.
__device__ double ms_digits_round(const unsigned long long* dig) {
  // carries: every digit becomes < 2^32; then five 64-bit limbs
  uint64_t L[5];
  unsigned long long c = 0ull;
  uint32_t d32[kMsDigits];
  for (int i = 0; i < kMsDigits; ++i) {
    const unsigned long long t = dig[i] + c;
    d32[i] = (uint32_t)t;
    c = t >> 32;
  }
  for (int i = 0; i < 5; ++i) L[i] = (uint64_t)d32[2 * i] | ((uint64_t)d32[2 * i + 1] << 32);
  int top = -1;
  for (int i = 4; i >= 0 && top < 0; --i)
    if (L[i]) top = 64 * i + 63 - __clzll((long long)L[i]);
  double v = 0.0;
  if (top >= 0 && top < 53) {
    v = ldexp((double)L[0], -149);
  } else if (top >= 53) {
    const int lo = top - 52, rb = lo - 1;
    auto bits64 = [&](int b) -> uint64_t {  // 64 bits of L from bit b
      const int q = b >> 6, o = b & 63;
      uint64_t x = L[q] >> o;
      if (o && q + 1 < 5) x |= L[q + 1] << (64 - o);
      return x;
    };
    uint64_t m = bits64(lo) & ((1ull << 53) - 1ull);
    const bool rnd = (bits64(rb) & 1ull) != 0ull;
    bool sticky = false;
    for (int i = 0; i < 5; ++i) {
      const int b0 = 64 * i;
      if (b0 + 64 <= rb) sticky |= L[i] != 0ull;
      else if (b0 < rb) sticky |= (L[i] & ((1ull << (rb - b0)) - 1ull)) != 0ull;
    }
    int e = lo;
    if (rnd && (sticky || (m & 1ull))) {
      ++m;
      if (m == (1ull << 53)) {
        m >>= 1;
        ++e;
      }
    }
    v = ldexp((double)m, e - 149);
  }
  return v;
}

// Significand (hidden bit included) of |x| added into its bin of the top
// 11 key bits (exponent field and three leading fraction bits: the same
// spread of addresses as a level-1 histogram, so few lanes of a wavefront
// collide). Infinities and NaNs are left out (they make the input invalid).
__device__ __forceinline__ void ms_accum(uint32_t key, unsigned long long* es) {
  const uint32_t E = key >> 23;
  const uint32_t m = (key & 0x7FFFFFu) | (E ? 0x800000u : 0u);
  if (E < 255u) atomicAdd(&es[key >> kH1Shift], (unsigned long long)m);
}

// Keys of the nb - 1 thresholds of the next log2(nb) rounds into K[] (LDS):
// ratio_j = l + j (r - l) / nb (exact: r - l is a power of two), thres_j =
// mean + ratio_j (u - mean) (the same double operations as a round of the
// loop). A pass that runs fewer rounds uses the nodes of the same grid that
// its rounds reach. Whole workgroup; ends with a barrier.
__device__ __forceinline__ double ms_step(const MsState& s, int nb) {
  return (s.r - s.l) * (1.0 / (double)nb);  // exact: both factors are powers of two
}
__device__ __forceinline__ uint32_t ms_key_at(const MsState& s, double step, int j) {
  const double ratio = s.l + step * (double)j;
  return ms_key_ceil(s.abar + ratio * (s.u - s.abar));
}
__device__ __forceinline__ void ms_keys(const MsState& s, uint32_t* K, int nb) {
  const double step = ms_step(s, nb);
  for (int j = threadIdx.x; j < nb; j += blockDim.x) K[j] = j ? ms_key_at(s, step, j) : 0u;
  __syncthreads();
}

// Bin of a key in a pass: the largest j with K[j] <= key (key >= K[1]; the
// keys ascend). K[8], K[16], .., K[56] first (seven reads in flight
// together), then the seven keys of that group of eight.
__device__ __forceinline__ int ms_bin(const uint32_t* K, uint32_t key) {
  int g = 0;
#pragma unroll
  for (int i = 1; i < 8; ++i) g += (K[8 * i] <= key) ? 1 : 0;
  const int base = 8 * g;
  int j = base;
#pragma unroll
  for (int i = 1; i < 8; ++i) j += (K[base + i] <= key) ? 1 : 0;
  return j;
}

// The same over the 4095 keys of a later pass: three levels of fifteen
// comparisons (K[256 i], then K[base + 16 i], then K[base + i]).
__device__ __forceinline__ int ms_bin_big(const uint32_t* K, uint32_t key) {
  static_assert(kMsRefineKeys == 4096, "three levels of 16");
  int base = 0;
#pragma unroll
  for (int lvl = 256; lvl >= 1; lvl >>= 4) {
    int g = 0;
#pragma unroll
    for (int i = 1; i < 16; ++i) g += (K[base + lvl * i] <= key) ? 1 : 0;
    base += lvl * g;
  }
  return base;
}

// The thresholds of a pass are evenly spaced in value: threshold j is
// abar + (l + j step)(u - abar). So the bin of a magnitude a is
// floor(((a - abar) / (u - abar) - l) / step) up to the roundings of that
// expression and of the thresholds' keys; ms_bin_est computes it in double
// and keeps it when its two keys bracket the element's key (one LDS round
// trip), else searches. Thresholds that round to one key (a narrow interval
// after a few passes) fail the check and are searched, so the result is
// always the search's.
struct MsEst {
  double c0, c1, c2;  // abar, 1 / ((u - abar) step), l / step
};
__device__ __forceinline__ MsEst ms_est(const MsState& s, int nb) {
  const double step = ms_step(s, nb);
  MsEst e;
  e.c0 = s.abar;
  e.c1 = 1.0 / ((s.u - s.abar) * step);  // (inf or NaN when u == abar: the check fails)
  e.c2 = s.l / step;
  return e;
}
__device__ __forceinline__ int ms_bin_est(const uint32_t* K, uint32_t key, const MsEst& e) {
  constexpr int NB = kMsRefineKeys;
  const double a = (double)__uint_as_float(key);
  double jd = floor((a - e.c0) * e.c1 - e.c2);
  jd = fmin(fmax(jd, 1.0), (double)(NB - 1));  // (fmax takes 1 over a NaN)
  const int j = (int)jd;
  const uint32_t lo = K[j];
  const uint32_t hi = (j + 1 < NB) ? K[j + 1] : 0xFFFFFFFFu;
  if (lo <= key && key < hi) return j;
  return ms_bin_big(K, key);
}
// The first pass: l = 0 and step = 1 / 64, so the bin is
// floor((a - abar) * 64 / (u - abar)); in binary32 (c0 = abar, c1 = 64 /
// (u - abar), both rounded), which the check makes exact all the same.
__device__ __forceinline__ int ms_bin_est64(const uint32_t* K, uint32_t key, float c0, float c1) {
  float jf = floorf((__uint_as_float(key) - c0) * c1);
  jf = fminf(fmaxf(jf, 1.0f), (float)(kMsKeys - 1));  // (fmaxf takes 1 over a NaN)
  const int j = (int)jf;
  const uint32_t lo = K[j];
  const uint32_t hi = (j + 1 < kMsKeys) ? K[j + 1] : 0xFFFFFFFFu;
  if (lo <= key && key < hi) return j;
  return ms_bin(K, key);
}

// The state before the first pass, from the stream's partial sums: nslots
// copies of the digits (kMsDigitStride words apart) and of the largest key.
// Whole workgroup (>= kMsDigits threads).
__device__ void ms_first_state(const unsigned long long* __restrict__ esum,
                               const uint32_t* __restrict__ emax, int nslots, int64_t d,
                               MsState& s, uint32_t* mk) {
  __shared__ unsigned long long dig[kMsDigits];
  const int tid = threadIdx.x;
  if (tid == 0) *mk = 0u;
  if (tid < kMsDigits) {
    unsigned long long v[kMsSlots];
#pragma unroll
    for (int sl = 0; sl < kMsSlots; ++sl)
      v[sl] = sl < nslots ? esum[(size_t)sl * kMsDigitStride + tid] : 0ull;
    unsigned long long t = 0ull;
#pragma unroll
    for (int sl = 0; sl < kMsSlots; ++sl) t += v[sl];
    dig[tid] = t;
  }
  __syncthreads();
  if (tid < nslots) atomicMax(mk, emax[tid]);
  __syncthreads();
  if (tid == 0) {
    const double total = ms_digits_round(dig);
    const uint32_t m = *mk;
    const bool bad = m >= 0x7F800000u;
    s.abar = bad ? 0.0 : total / (double)d;
    s.u = bad ? 0.0 : (double)__uint_as_float(m);
    s.l = 0.0;
    s.r = 1.0;
    s.k1 = 0u;
    s.k2 = (uint32_t)d;
    s.K1 = kMsNone;
    s.K2 = 0u;
    s.rand = 0u;
    s.take = 0u;
    s.level = 0u;
    s.bad = bad ? 1u : 0u;
  }
  __syncthreads();
}

// The state after a pass: its counts (nslots copies of nb bins, summed),
// suffix sums, and its rounds replayed (round i takes bin j = midpoint of
// the bins still open, whose ratio l + (r - l) / 2 equals l0 + j (r0 - l0) /
// nb exactly, so its threshold and key are the ones the pass counted
// against; the replay itself only moves bin indices and forms the keys of
// the recorded counts at the end). After round n_search the window offset
// and length are fixed too. Whole workgroup of kSBlock threads. h: nb words
// of LDS (64 or 4096).
__device__ void ms_next_state(const MsState& prev, const uint32_t* __restrict__ cnt, int nslots,
                              int nb, int32_t rounds, int32_t n_search, uint32_t k, int64_t d,
                              uint64_t window_word, MsState& s, uint32_t* h, uint32_t* wsum) {
  const int tid = threadIdx.x;
  for (int i = tid; i < nb; i += kSBlock) h[i] = 0u;
  __syncthreads();
  for (int i = tid; i < nslots * nb; i += kSBlock) {
    const uint32_t c = cnt[i];
    if (c) atomicAdd(&h[i & (nb - 1)], c);
  }
  __syncthreads();
  // nnz[j] = elements with key >= K[j] = sum of h[j..nb-1]
  if (nb == kMsKeys) {
    // the first wavefront, lane t holding bin 63 - t
    if (tid < 64) {
      const uint32_t run = wave_incl_scan(h[63 - tid]);
      __builtin_amdgcn_wave_barrier();
      h[63 - tid] = run;
    }
  } else {
    // thread t owns the four bins 4095 - 4t .. 4092 - 4t (from the top)
    static_assert(kMsRefineKeys == 4 * kSBlock, "four bins per thread");
    const int b0 = kMsRefineKeys - 4 * (tid + 1);
    uint32_t c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) c[q] = h[b0 + 3 - q];  // c[0] = highest bin
    uint32_t tot;
    const uint32_t ex = sblock_scan(c[0] + c[1] + c[2] + c[3], wsum, &tot);
    uint32_t run = ex;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      run += c[q];
      h[b0 + 3 - q] = run;
    }
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t k1 = prev.k1, k2 = prev.k2, K1 = prev.K1, K2 = prev.K2;
    int jl = 0, jh = nb, j1 = -1, j2 = -1;
    for (int i = 0; i < rounds; ++i) {
      const int j = (jl + jh) >> 1;
      const uint32_t n = h[j];
      if (n <= k) {
        jh = j;
        if (n > k1) {
          k1 = n;
          j1 = j;
        }
      } else {
        jl = j;
        if (n < k2) {
          k2 = n;
          j2 = j;
        }
      }
    }
    const double step = ms_step(prev, nb);
    if (j1 >= 0) K1 = ms_key_at(prev, step, j1);
    if (j2 >= 0) K2 = ms_key_at(prev, step, j2);
    const double l = prev.l + step * (double)jl, r = prev.l + step * (double)jh;
    s = prev;
    s.level = prev.level + (uint32_t)rounds;
    if (s.level >= (uint32_t)n_search) {
      if (prev.bad) {  // non-finite input: the first k positions
        k1 = 0u;
        k2 = (uint32_t)d;
        K1 = kMsNone;
        K2 = 0u;
        s.rand = 0u;
      } else {
        // band = k2 - k1 elements, k - k1 taken from it: offsets 0 .. k2 - k
        s.rand = (uint32_t)(window_word % ((uint64_t)(k2 - k) + 1ull));
      }
      s.take = k - k1;
    }
    s.l = l;
    s.r = r;
    s.k1 = k1;
    s.k2 = k2;
    s.K1 = K1;
    s.K2 = K2;
  }
  __syncthreads();
}

}  // namespace

__global__ __launch_bounds__(kBlock) void k_ms_stream(const TileDesc* __restrict__ tiles,
                                                      int32_t ntiles, int nslots,
                                                      unsigned long long* __restrict__ esum,
                                                      uint32_t* __restrict__ emax,
                                                      uint16_t* __restrict__ summ,
                                                      uint32_t* __restrict__ clear,
                                                      int64_t clear_words) {
  __shared__ unsigned long long es[kH1Bins];
  __shared__ unsigned long long dig[kMsDigits];
  __shared__ uint32_t bmax;
  const int tid = threadIdx.x;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + tid; i < clear_words;
       i += (int64_t)gridDim.x * kBlock)
    clear[i] = 0u;  // (as in k_stream)
  for (int i = tid; i < kH1Bins; i += kBlock) es[i] = 0ull;
  if (tid < kMsDigits) dig[tid] = 0ull;
  if (tid == 0) bmax = 0u;
  __syncthreads();
  const int slot = blockIdx.x % nslots;
  const int nunits = ntiles * (kTile / kQuarter);
  uint32_t tmax = 0u;
  for (int unit = blockIdx.x; unit < nunits; unit += gridDim.x) {
    const TileDesc t = tiles[unit / (kTile / kQuarter)];
    const int s0 = (unit % (kTile / kQuarter)) * kQuarter;
    if (s0 >= t.len) continue;
    const int len = min(kQuarter, t.len - s0);
    const float* __restrict__ g = t.g + s0;
    float* __restrict__ r = t.r + s0;
    uint16_t* __restrict__ sq = summ + (size_t)(unit / (kTile / kQuarter)) * kLinesPerTile +
                                s0 / kLine;
    const bool full = len == kQuarter &&
        ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(r)) & 15u) == 0;
    if (full) {
      const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
      float4* __restrict__ r4 = reinterpret_cast<float4*>(r);
      float4 a[kQV], b[kQV];
#pragma unroll
      for (int v = 0; v < kQV; ++v) a[v] = load_nt4(g4 + v * kBlock + tid);
#pragma unroll
      for (int v = 0; v < kQV; ++v) b[v] = load_nt4(r4 + v * kBlock + tid);
#pragma unroll
      for (int v = 0; v < kQV; ++v) {
        float4 x;
        x.x = a[v].x + b[v].x;
        x.y = a[v].y + b[v].y;
        x.z = a[v].z + b[v].z;
        x.w = a[v].w + b[v].w;
        store_nt4(r4 + v * kBlock + tid, x);
        const uint32_t k0 = mag_key(x.x), k1 = mag_key(x.y), k2 = mag_key(x.z), k3 = mag_key(x.w);
        ms_accum(k0, es);
        ms_accum(k1, es);
        ms_accum(k2, es);
        ms_accum(k3, es);
        uint32_t m = max(max(k0, k1), max(k2, k3));
        tmax = max(tmax, m);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        m = max(m, (uint32_t)__shfl_xor((int)m, 4));
        if ((tid & 7) == 0) sq[(v * kBlock + tid) >> 3] = (uint16_t)(m >> 16);
      }
    } else {
      // partial or misaligned quarter, as in k_stream: element by element,
      // line maxima reduced over the 32 lanes that hold each line
      constexpr int kPer = kQuarter / kBlock;
      float gv[kPer], rv[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        gv[q] = (e < len) ? __builtin_nontemporal_load(gptr(g) + e) : 0.0f;
        rv[q] = (e < len) ? __builtin_nontemporal_load(gptr(r) + e) : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * kBlock + tid;
        uint32_t k = 0u;
        if (e < len) {
          const float x = gv[q] + rv[q];
          __builtin_nontemporal_store(x, gptr(r) + e);
          k = mag_key(x);
          ms_accum(k, es);
          tmax = max(tmax, k);
        }
        k = max(k, (uint32_t)__shfl_xor((int)k, 1));
        k = max(k, (uint32_t)__shfl_xor((int)k, 2));
        k = max(k, (uint32_t)__shfl_xor((int)k, 4));
        k = max(k, (uint32_t)__shfl_xor((int)k, 8));
        k = max(k, (uint32_t)__shfl_xor((int)k, 16));
        if ((tid & (kLine - 1)) == 0 && e < len) sq[e / kLine] = (uint16_t)(k >> 16);
      }
    }
  }
  atomicMax(&bmax, tmax);
  __syncthreads();
  // thread E: the eight bins of exponent field E, as digits of this
  // workgroup's exact sum, which are then added into this copy
  static_assert(kBlock == 256 && kH1Bins == 8 * kBlock, "one exponent per thread");
  unsigned long long v = 0ull;
#pragma unroll
  for (int i = 0; i < 8; ++i) v += es[8 * tid + i];
  if (tid < 255) ms_digits_add(tid, v, dig);
  __syncthreads();
  if (tid < kMsDigits && dig[tid]) atomicAdd(&esum[(size_t)slot * kMsDigitStride + tid], dig[tid]);
  if (tid == 0 && bmax) atomicMax(&emax[slot], bmax);
}

// First counting pass: the state before it (mean, u), then every element
// against the 63 keys of rounds 1..6 (persistent grid of kBlock-thread
// workgroups walking units of kQuarter elements, two units in flight). A
// line whose summary is below the lowest key holds no element to count and
// is not read. A thread's hits (key >= lowest key) are marked in a bit mask
// and binned one per round, so a wavefront runs as many bin searches as its
// busiest lane has hits.
__global__ __launch_bounds__(kBlock) void k_ms_count(
    const TileDesc* __restrict__ tiles, int32_t ntiles, int nslots,
    const unsigned long long* __restrict__ esum, const uint32_t* __restrict__ emax,
    const uint16_t* __restrict__ summ, uint32_t* __restrict__ cnt,
    MsState* __restrict__ st_out, int64_t d, uint32_t* __restrict__ status) {
  __shared__ MsState s;
  __shared__ uint32_t K[kMsKeys];
  __shared__ uint32_t h[kMsKeys];
  __shared__ uint32_t mk;
  const int tid = threadIdx.x;
  ms_first_state(esum, emax, nslots, d, s, &mk);
  if (blockIdx.x == 0 && tid == 0) {
    *st_out = s;
    if (s.bad && status) atomicOr(status, TKEF_STATUS_NONFINITE);
  }
  if (tid < kMsKeys) h[tid] = 0u;
  ms_keys(s, K, kMsKeys);
  // (the first pass brackets the ratio in [0, 1])
  const float c0 = (float)s.abar, c1 = (float)(64.0 / (s.u - s.abar));
  const uint32_t kmin = K[1];
  const uint32_t smin = kmin >> 16;  // a line is read if its summary reaches this
  const int per_tile = kTile / kQuarter;
  const int nunits = ntiles * per_tile;
  constexpr int kSlots = 2 * kQV * 4;  // elements per thread per iteration
  static_assert(kSlots <= 32, "hit mask");
  for (int u0 = blockIdx.x; u0 < nunits; u0 += 2 * gridDim.x) {
    float4 f[2][kQV];
    int len[2];
    bool full[2];
    const float* xs[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int unit = u0 + q * gridDim.x;
      len[q] = 0;
      full[q] = false;
      xs[q] = nullptr;
      if (unit < nunits) {
        const int tile = unit / per_tile;
        const int s0 = (unit % per_tile) * kQuarter;
        // the summaries' address does not depend on the descriptor: both
        // loads are issued together
        const uint16_t* sq = summ + (size_t)tile * kLinesPerTile + s0 / kLine;
        uint32_t sv[kQV];
#pragma unroll
        for (int v = 0; v < kQV; ++v) sv[v] = sq[(v * kBlock + tid) >> 3];
        const TileDesc t = tiles[tile];
        len[q] = s0 < t.len ? min(kQuarter, t.len - s0) : 0;
        xs[q] = t.r + s0;
        full[q] = len[q] == kQuarter && (reinterpret_cast<uintptr_t>(xs[q]) & 15u) == 0;
        if (full[q]) {
          const float4* x4 = reinterpret_cast<const float4*>(xs[q]);
#pragma unroll
          for (int v = 0; v < kQV; ++v) {
            const int i4 = v * kBlock + tid;  // float4 index: line i4 / 8
            f[q][v] = (sv[v] >= smin) ? load_nt4(x4 + i4) : make_float4(0.f, 0.f, 0.f, 0.f);
          }
        }
      }
    }
    uint32_t keys[kSlots];
    uint32_t hits = 0u;
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int v = 0; v < kQV; ++v) {
        const int b = (q * kQV + v) * 4;
        keys[b + 0] = mag_key(f[q][v].x);
        keys[b + 1] = mag_key(f[q][v].y);
        keys[b + 2] = mag_key(f[q][v].z);
        keys[b + 3] = mag_key(f[q][v].w);
#pragma unroll
        for (int c = 0; c < 4; ++c)
          hits |= (full[q] && keys[b + c] >= kmin) ? (1u << (b + c)) : 0u;
      }
#pragma unroll 1
    while (hits) {
      const int j = __ffs(hits) - 1;
      hits &= hits - 1u;
      uint32_t key = 0u;
#pragma unroll
      for (int c = 0; c < kSlots; ++c) key = (c == j) ? keys[c] : key;
      atomicAdd(&h[ms_bin_est64(K, key, c0, c1)], 1u);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (!full[q] && len[q] > 0) {
        for (int e = tid; e < len[q]; e += kBlock) {
          const uint32_t key = mag_key(gptr(xs[q])[e]);
          if (key >= kmin) atomicAdd(&h[ms_bin_est64(K, key, c0, c1)], 1u);
        }
      }
    }
  }
  __syncthreads();
  const int slot = blockIdx.x % nslots;
  if (tid < kMsKeys && h[tid]) atomicAdd(&cnt[(size_t)slot * kMsKeys + tid], h[tid]);
}

// Later counting passes: the state after the previous pass, then the lines
// whose summary reaches keys[1] (the lowest threshold left to try), counted
// against 4095 keys (up to twelve rounds), read by the selection regions.
// The previous pass left prev_slots copies of prev_nb bins; this pass adds
// into one copy of 4096.
__global__ __launch_bounds__(kSBlock) void k_ms_refine(
    const TileDesc* __restrict__ tiles, const uint16_t* __restrict__ summ, int64_t nlines,
    int lpt, int prev_slots, int prev_nb, const uint32_t* __restrict__ cnt_prev,
    uint32_t* __restrict__ cnt, const MsState* __restrict__ st_prev, MsState* __restrict__ st_out,
    uint32_t k, int64_t d, int32_t rounds_prev, int32_t n_search, uint64_t window_word) {
  __shared__ MsState s;
  __shared__ uint32_t K[kMsRefineKeys];
  __shared__ uint32_t h[kMsRefineKeys];
  __shared__ uint32_t wsum[kSWaves];
  const int tid = threadIdx.x;
  // this thread's summaries first: their latency overlaps the state
  LineSpan ls;
  ls.load(tiles, summ, nlines, ((int64_t)blockIdx.x * kSBlock + tid) * lpt, lpt);
  const MsState prev = *st_prev;
  ms_next_state(prev, cnt_prev, prev_slots, prev_nb, rounds_prev, n_search, k, d, window_word, s,
                h, wsum);
  if (blockIdx.x == 0 && tid == 0) *st_out = s;
  for (int i = tid; i < kMsRefineKeys; i += kSBlock) h[i] = 0u;
  ms_keys(s, K, kMsRefineKeys);
  const MsEst est = ms_est(s, kMsRefineKeys);
  const uint32_t kmin = K[1];
  const uint32_t mask = ls.flagged([&](int) -> uint32_t { return kmin; });
  walk_mask(ls, mask, [&](int, uint32_t key) -> bool { return key >= kmin; },
            [&](int, const TileDesc&, int, float, uint32_t key) {
              atomicAdd(&h[ms_bin_est(K, key, est)], 1u);
            });
  __syncthreads();
  for (int i = tid; i < kMsRefineKeys; i += kSBlock)
    if (h[i]) atomicAdd(&cnt[i], h[i]);
}

// Ordered compaction: an element with key >= K1 goes to slot (#key >= K1
// before it) + (#window members before it); a band member (K2 <= key < K1)
// whose rank in the band lies in [rand, rand + take) goes to slot (#key >= K1
// before it) + rank - rand. Prefixes across workgroups come from a bounded
// look-back over the regions before.
__global__ __launch_bounds__(kSBlock) void k_ms_emit(
    const TileDesc* __restrict__ tiles, const uint16_t* __restrict__ summ, int64_t nlines,
    int lpt, int prev_slots, int prev_nb, const uint32_t* __restrict__ cnt_prev,
    const MsState* __restrict__ st_prev, MsState* __restrict__ st_out, uint32_t k, int64_t d,
    int32_t rounds_prev, int32_t n_search, uint64_t window_word, uint64_t* __restrict__ flags,
    int32_t* __restrict__ idx_out, void* __restrict__ val_out, int val16,
    uint32_t* __restrict__ status, uint32_t* __restrict__ clear_next, int64_t clear_words) {
  __shared__ MsState s;
  __shared__ uint32_t h[kMsRefineKeys];
  __shared__ uint32_t wsum[2 * kSWaves];
  __shared__ uint64_t red[kSWaves];
  __shared__ int32_t stage_code[kStage * kSBlock];
  __shared__ float stage_x[kStage * kSBlock];
  const int tid = threadIdx.x;
  // this thread's summaries first: their latency overlaps the state
  LineSpan ls;
  ls.load(tiles, summ, nlines, ((int64_t)blockIdx.x * kSBlock + tid) * lpt, lpt);
  const MsState prev = *st_prev;
  ms_next_state(prev, cnt_prev, prev_slots, prev_nb, rounds_prev, n_search, k, d, window_word, s,
                h, wsum);
  if (blockIdx.x == 0 && tid == 0) *st_out = s;
#pragma unroll 1
  for (int64_t i = (int64_t)blockIdx.x * kSBlock + tid; i < clear_words;
       i += (int64_t)gridDim.x * kSBlock)
    clear_next[i] = 0u;
  const uint32_t K1 = s.K1, K2 = s.K2, rand = s.rand, take = s.take;
  const uint32_t mask = ls.flagged([&](int) -> uint32_t { return K2; });
  auto hit = [&](int, uint32_t key) -> bool { return key >= K2; };
  uint32_t c1 = 0u, c2 = 0u, nst = 0u;
  walk_mask(ls, mask, hit, [&](int tile, const TileDesc&, int e, float x, uint32_t key) {
    if (nst < (uint32_t)kStage) {
      stage_code[nst * kSBlock + tid] = (int32_t)(((uint32_t)tile << kCandShift) | (uint32_t)e);
      stage_x[nst * kSBlock + tid] = x;
    }
    ++nst;
    if (key >= K1) ++c1;
    else ++c2;
  });
  uint2 tot;
  const uint2 ex = block_scan2<kSBlock>(c1, c2, wsum, &tot);
  bool ok;
  const uint64_t pre =
      group_prefix(flags, (uint64_t)tot.x | ((uint64_t)tot.y << 31), red, status, &ok);
  if (nst == 0u || !ok) return;  // (no place is known without the full prefix)
  uint32_t p1 = (uint32_t)(pre & 0x7FFFFFFFu) + ex.x;
  uint32_t p2 = (uint32_t)((pre >> 31) & 0x7FFFFFFFu) + ex.y;
  auto write = [&](int, const TileDesc& t, int e, float x, uint32_t key) {
    uint32_t pos = 0xFFFFFFFFu;
    if (key >= K1) {
      pos = p1 + min(p2 > rand ? p2 - rand : 0u, take);
      ++p1;
    } else {
      if (p2 >= rand && p2 - rand < take) pos = p1 + (p2 - rand);
      ++p2;
    }
    if (pos < k) {
      idx_out[pos] = t.gstart + e;
      put_val(val_out, (size_t)pos, x, val16);
      gptr(t.r)[e] = 0.0f;
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
  } else {
    walk_mask(ls, mask, hit, write);
  }
}

// ---------------------------------------------------------------------------
// Fixed scratch for the entry point that allocates nothing: one array per
// GPU, in the library's device memory until the process ends. Host code
// never passes the array's name to a kernel (on the host it only names a
// stand-in); it uses the address hipGetSymbolAddress returns for the current
// device, kept per device.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

void* static_scratch(hipError_t* err) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && (dev < 0 || dev >= kMaxDevices)) e = hipErrorInvalidDevice;
  if (e != hipSuccess) {
    *err = e;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    addr[dev] = ptr;
  }
  *err = hipSuccess;
  return addr[dev];
}

// The descriptors of one tensor (what bind copies from the host for a plan)
// and the words that must start at zero.
__global__ void k_setup_one(TileDesc* __restrict__ tiles, GroupDesc* __restrict__ groups,
                            const float* g, float* r, int64_t d, int64_t k, int32_t ntiles,
                            uint32_t* __restrict__ zero, int64_t n_zero,
                            uint32_t* __restrict__ tail, int64_t n_tail) {
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < ntiles; i += step) {
    TileDesc t;
    t.g = g + i * kTile;
    t.r = r + i * kTile;
    t.gstart = (int32_t)(i * kTile);
    t.len = (int32_t)min((int64_t)kTile, d - i * kTile);
    t.group = 0;
    t.reserved = 0;
    tiles[i] = t;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) groups[0] = GroupDesc{(uint32_t)k, 0u, 0u, 0u};
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_zero; i += step)
    zero[i] = 0u;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_tail; i += step)
    tail[i] = 0u;
}

// ---------------------------------------------------------------------------
// launchers (the timing events, when given, are recorded by the dispatch)

template <typename K, typename... Args>
hipError_t launch(K kernel, dim3 grid, dim3 block, hipStream_t s, const Ev& ev, Args... args) {
  hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev.start, ev.stop, 0, args...);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  return launch(k_fill_u32, dim3((unsigned)blocks), dim3(256), s, Ev{}, p, v, n);
}

hipError_t launch_setup_one(TileDesc* tiles, GroupDesc* groups, const float* g, float* r,
                            int64_t d, int64_t k, int32_t ntiles, uint32_t* zero, int64_t n_zero,
                            uint32_t* tail, int64_t n_tail, hipStream_t s) {
  int64_t n = ntiles;
  if (n_zero > n) n = n_zero;
  if (n_tail > n) n = n_tail;
  int64_t blocks = (n + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 1024) blocks = 1024;
  return launch(k_setup_one, dim3((unsigned)blocks), dim3(256), s, Ev{}, tiles, groups, g, r, d,
                k, ntiles, zero, n_zero, tail, n_tail);
}

hipError_t launch_stream(const TileDesc* tiles, int32_t ntiles, int32_t grid, uint32_t* hist1,
                         int32_t nslots, uint16_t* summ, uint32_t* status, uint32_t* clear,
                         int64_t clear_words, hipStream_t s, const Ev& ev) {
  return launch(k_stream, dim3(grid), dim3(kBlock), s, ev, tiles, ntiles, hist1, nslots, summ,
                status, clear, clear_words);
}

hipError_t launch_pick(int level, const GroupDesc* groups, GroupState* st,
                       const uint32_t* hist, int32_t nslots, int32_t ngroups, hipStream_t s,
                       const Ev& ev) {
  static_assert(kH1Bins == 8 * kBlock && kH2Bins == 4 * kBlock && kH3Bins == 4 * kBlock,
                "pick: bins per thread");
  if (level == 1) {
    if (nslots != kSlotsMany) return hipErrorInvalidValue;
    return launch(k_pick<8, kSlotsMany>, dim3(ngroups), dim3(kBlock), s, ev, level, groups, st,
                  hist);
  }
  if (nslots != 1) return hipErrorInvalidValue;
  return launch(k_pick<4, 1>, dim3(ngroups), dim3(kBlock), s, ev, level, groups, st, hist);
}

hipError_t launch_collect(const TileDesc* tiles, const GroupDesc* groups, GroupState* st,
                          const uint32_t* hist1, int nslots, const uint16_t* summ, int64_t nlines,
                          int lpt, int32_t grid, int32_t block, uint32_t rcap, uint32_t* hist2, uint32_t* rbin,
                          uint32_t* rcand, uint32_t* rband, uint32_t* rbtmp, uint32_t* rsuf,
                          uint32_t* rcnt, hipStream_t s, const Ev& ev) {
  if (nslots != kSlotsOne) return hipErrorInvalidValue;
  if (block == kCBlockSmall)
    return launch(k_collect<kCBlockSmall>, dim3(grid), dim3(block), s, ev, tiles, groups, st,
                  hist1, summ, hist2, rbin, reinterpret_cast<uint4*>(rcand), rband, rbtmp, rsuf,
                  reinterpret_cast<uint2*>(rcnt), rcap, lpt, nlines);
  if (block == kSBlock)
    return launch(k_collect<kSBlock>, dim3(grid), dim3(block), s, ev, tiles, groups, st, hist1,
                  summ, hist2, rbin, reinterpret_cast<uint4*>(rcand), rband, rbtmp, rsuf,
                  reinterpret_cast<uint2*>(rcnt), rcap, lpt, nlines);
  return hipErrorInvalidValue;
}

hipError_t launch_finish(const TileDesc* tiles, const GroupDesc* groups,
                         const GroupState* st, const uint16_t* summ, int64_t nlines, int lpt,
                         int32_t grid, int32_t block, uint32_t rcap, const uint32_t* hist2, const uint32_t* rbin,
                         const uint32_t* rcand, const uint32_t* rband, const uint32_t* rsuf,
                         const uint32_t* rcnt, int32_t* idx_out, void* val_out, int val16,
                         uint32_t* clear_next, int64_t clear_words, uint32_t* ticket,
                         uint32_t* rzr, hipStream_t s, const Ev& ev) {
  uint64_t* rz = reinterpret_cast<uint64_t*>(rzr);
  if (block == kCBlockSmall)
    return launch(k_finish<kCBlockSmall>, dim3(grid), dim3(block), s, ev, tiles, groups, st, summ,
                  nlines, lpt, rcap, hist2, rbin, reinterpret_cast<const uint4*>(rcand), rband,
                  rsuf, reinterpret_cast<const uint2*>(rcnt), idx_out, val_out, val16,
                  clear_next, clear_words, ticket, rz);
  if (block == kSBlock)
    return launch(k_finish<kSBlock>, dim3(grid), dim3(block), s, ev, tiles, groups, st, summ,
                  nlines, lpt, rcap, hist2, rbin, reinterpret_cast<const uint4*>(rcand), rband,
                  rsuf, reinterpret_cast<const uint2*>(rcnt), idx_out, val_out, val16,
                  clear_next, clear_words, ticket, rz);
  return hipErrorInvalidValue;
}

hipError_t launch_gather(const TileDesc* tiles, const GroupState* st, const uint16_t* summ,
                         int64_t nlines, int lpt, int32_t grid, uint32_t* hist2, uint64_t* flags,
                         uint32_t* cand, uint32_t cap, uint32_t* meta, uint32_t* status,
                         hipStream_t s, const Ev& ev) {
  return launch(k_gather, dim3(grid), dim3(kSBlock), s, ev, tiles, st, summ, nlines, lpt, hist2,
                flags, reinterpret_cast<uint2*>(cand), cap, meta, status);
}

hipError_t launch_hist3(const TileDesc* tiles, int32_t ntiles, const GroupState* st,
                        const uint16_t* summ, int64_t nlines, int lpt, int32_t grid,
                        const uint32_t* cand, const uint32_t* meta, uint32_t* hist3,
                        hipStream_t s, const Ev& ev) {
  return launch(k_hist3, dim3(grid), dim3(kSBlock), s, ev, tiles, ntiles, st, summ, nlines, lpt,
                reinterpret_cast<const uint2*>(cand), meta, hist3);
}

hipError_t launch_groupscan(const GroupDesc* groups, const GroupState* st, int32_t ngroups,
                            uint32_t* base, hipStream_t s, const Ev& ev) {
  return launch(k_groupscan, dim3(1), dim3(kSBlock), s, ev, groups, st, ngroups, base);
}

hipError_t launch_emit(const TileDesc* tiles, int32_t ntiles, const GroupDesc* groups,
                       const GroupState* st, const uint16_t* summ, int64_t nlines, int lpt,
                       int32_t grid, const uint32_t* cand, const uint32_t* meta,
                       const uint32_t* base, uint64_t* flags, int32_t* idx_out, void* val_out,
                       int val16, uint32_t* status, uint32_t* clear_next, int64_t clear_words,
                       int32_t fold_ngroups, hipStream_t s, const Ev& ev) {
  if (fold_ngroups > kEmitLdsGroups) return hipErrorInvalidValue;
  // (one instantiation per case, so that no load picks between an LDS and a
  // global address at run time: that would be a flat load)
  return launch(fold_ngroups > 0 ? k_emit<true> : k_emit<false>, dim3(grid), dim3(kSBlock), s, ev,
                tiles, ntiles, groups, st, summ, nlines,
                lpt, reinterpret_cast<const uint2*>(cand), meta, base, flags, idx_out, val_out,
                val16, status, clear_next, clear_words, fold_ngroups);
}

hipError_t launch_ms_stream(const TileDesc* tiles, int32_t ntiles, int32_t grid, int32_t nslots,
                            uint64_t* esum, uint32_t* emax, uint16_t* summ, uint32_t* clear,
                            int64_t clear_words, hipStream_t s, const Ev& ev) {
  return launch(k_ms_stream, dim3(grid), dim3(kBlock), s, ev, tiles, ntiles, (int)nslots,
                reinterpret_cast<unsigned long long*>(esum), emax, summ, clear, clear_words);
}

hipError_t launch_ms_count(const TileDesc* tiles, int32_t ntiles, int32_t grid, int32_t nslots,
                           const uint64_t* esum, const uint32_t* emax, const uint16_t* summ,
                           uint32_t* cnt, MsState* st_out, int64_t d, uint32_t* status,
                           hipStream_t s, const Ev& ev) {
  return launch(k_ms_count, dim3(grid), dim3(kBlock), s, ev, tiles, ntiles, (int)nslots,
                reinterpret_cast<const unsigned long long*>(esum), emax, summ, cnt, st_out, d,
                status);
}

hipError_t launch_ms_refine(const TileDesc* tiles, const uint16_t* summ, int64_t nlines, int lpt,
                            int32_t grid, int32_t prev_slots, int32_t prev_nb,
                            const uint32_t* cnt_prev, uint32_t* cnt, const MsState* st_prev,
                            MsState* st_out, uint32_t k, int64_t d, int32_t rounds_prev,
                            int32_t n_search, uint64_t window_word, hipStream_t s,
                            const Ev& ev) {
  return launch(k_ms_refine, dim3(grid), dim3(kSBlock), s, ev, tiles, summ, nlines, lpt,
                (int)prev_slots, (int)prev_nb, cnt_prev, cnt, st_prev, st_out, k, d, rounds_prev,
                n_search, window_word);
}

hipError_t launch_ms_emit(const TileDesc* tiles, const uint16_t* summ, int64_t nlines, int lpt,
                          int32_t grid, int32_t prev_slots, int32_t prev_nb,
                          const uint32_t* cnt_prev, const MsState* st_prev, MsState* st_out,
                          uint32_t k, int64_t d, int32_t rounds_prev, int32_t n_search,
                          uint64_t window_word, uint64_t* flags, int32_t* idx_out,
                          void* val_out, int val16, uint32_t* status, uint32_t* clear_next,
                          int64_t clear_words, hipStream_t s, const Ev& ev) {
  return launch(k_ms_emit, dim3(grid), dim3(kSBlock), s, ev, tiles, summ, nlines, lpt,
                (int)prev_slots, (int)prev_nb, cnt_prev, st_prev, st_out, k, d, rounds_prev,
                n_search, window_word, flags, idx_out, val_out, val16, status, clear_next,
                clear_words);
}

int32_t select_max_groups() { return kSMaxGroups; }
int32_t select_block() { return kSBlock; }
int32_t collect_block(int64_t nlines, int64_t k, int64_t d) {
  const bool fits = nlines <= (int64_t)kCBlockSmall * kSMaxLpt * kCDenseMaxGroups;
  return (nlines <= kCSmallLines || (k * kCDenseDiv >= d && fits)) ? kCBlockSmall : kSBlock;
}
int32_t select_max_lpt() { return kSMaxLpt; }
int32_t emit_lds_groups() { return kEmitLdsGroups; }

hipError_t launch_seg(const int32_t* idx, int64_t stride, const int32_t* nnz, int32_t P,
                      int32_t d, int32_t ntiles_u, int32_t* seg, uint32_t* status,
                      hipStream_t s, const Ev& ev) {
  int64_t bx = (stride + 255) / 256;
  if (bx < 1) bx = 1;
  const ListsArg lists{idx, nullptr, stride, nnz, nullptr};
  return launch(k_seg<false>, dim3((unsigned)bx, (unsigned)P), dim3(256), s, ev, lists, P, d,
                ntiles_u, seg, status);
}

hipError_t launch_seg_table(const WorkerList* table, int32_t P, int64_t max_n, int32_t d,
                            int32_t ntiles_u, int32_t* seg, uint32_t* status, hipStream_t s,
                            const Ev& ev) {
  int64_t bx = (max_n + 255) / 256;
  if (bx < 1) bx = 1;
  const ListsArg lists{nullptr, nullptr, 0, nullptr, table};
  return launch(k_seg<true>, dim3((unsigned)bx, (unsigned)P), dim3(256), s, ev, lists, P, d,
                ntiles_u, seg, status);
}

// whole groups of kXcds runs (workgroups past the last tile return at once)
static int32_t update_grid(int32_t ntiles_u) {
  constexpr int32_t kGroup = kXcds * kXcdRun;
  return (ntiles_u + kGroup - 1) / kGroup * kGroup;
}

hipError_t launch_update(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                         int32_t d, int32_t ntiles_u, const int32_t* idx, const void* val,
                         int val16, int64_t stride, const int32_t* nnz, int32_t P,
                         const int32_t* seg, float lr, float mu, float wd, int op, int has_mom,
                         const LarsArgs& lars, bool det, hipStream_t s, const Ev& ev) {
  const bool is_lars = op == kOpLarsNorm || op == kOpLarsApply;
  const ListsArg lists{idx, val, stride, nnz, nullptr};
  auto* kern = is_lars ? (det ? k_update<true, false, true> : k_update<true, false, false>)
                       : (det ? k_update<false, false, true> : k_update<false, false, false>);
  return launch(kern,
                dim3(update_grid(ntiles_u)), dim3(kUBlock), s, ev, tens, tile_first, ntens, d,
                ntiles_u, lists, val16, P, seg, lr, mu, wd, op, has_mom, lars);
}

hipError_t launch_update_table(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                               int32_t d, int32_t ntiles_u, const WorkerList* table, int32_t P,
                               const int32_t* seg, float lr, float mu, float wd, int op,
                               int has_mom, hipStream_t s, const Ev& ev) {
  const ListsArg lists{nullptr, nullptr, 0, nullptr, table};
  return launch(k_update<false, true, false>, dim3(update_grid(ntiles_u)), dim3(kUBlock), s, ev, tens,
                tile_first, ntens, d, ntiles_u, lists, 0, P, seg, lr, mu, wd, op, has_mom,
                LarsArgs{nullptr, nullptr, nullptr, 0.0f});
}

hipError_t launch_lars_norm_dense(const UpdTensor* tens, const float* const* gptrs,
                                  const int32_t* tile_first, int32_t ntens, int32_t d,
                                  int32_t ntiles_u, double2* part, const int32_t* tpair,
                                  hipStream_t s, const Ev& ev) {
  return launch(k_lars_norm_dense, dim3(ntiles_u), dim3(kUBlock), s, ev, tens, gptrs, tile_first,
                ntens, d, ntiles_u, part, tpair);
}

hipError_t launch_lars_rates(const int32_t* tpair, const double2* part, int32_t ntens,
                             double gamma, double eta, double eps, double* rate,
                             double* rate_out, hipStream_t s, const Ev& ev) {
  return launch(k_lars_rates, dim3(ntens), dim3(kUBlock), s, ev, tpair, part, gamma, eta, eps,
                rate, rate_out);
}

}  // namespace tkef

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
__device__ __forceinline__ void stream_quad(float4 a, float4 b, float4& x, uint32_t* h,
                                            uint32_t& m) {
  x.x = a.x + b.x;
  x.y = a.y + b.y;
  x.z = a.z + b.z;
  x.w = a.w + b.w;
  const uint32_t k0 = mag_key(x.x), k1 = mag_key(x.y), k2 = mag_key(x.z),
                 k3 = mag_key(x.w);
  atomicAdd(&h[k0 >> kH1Shift], 1u);
  atomicAdd(&h[k1 >> kH1Shift], 1u);
  atomicAdd(&h[k2 >> kH1Shift], 1u);
  atomicAdd(&h[k3 >> kH1Shift], 1u);
  m = max(max(k0, k1), max(k2, k3));
}

__global__ __launch_bounds__(kBlock) void k_stream(const TileDesc* __restrict__ tiles,
                                                   uint32_t* __restrict__ hist1,
                                                   uint16_t* __restrict__ summ,
                                                   uint32_t* __restrict__ status) {
  __shared__ uint32_t h[kH1Bins];
  __shared__ uint32_t lmax[kLinesPerTile];
  __shared__ uint32_t nanflag;
  const int tid = threadIdx.x;
  const TileDesc t = tiles[blockIdx.x];
  for (int i = tid; i < kH1Bins; i += kBlock) h[i] = 0u;
  lmax[tid] = 0u;
  if (tid == 0) nanflag = 0u;
  __syncthreads();

  const int len = t.len;
  const float* __restrict__ g = t.g;
  float* __restrict__ r = t.r;
  uint32_t tmax = 0u;  // largest key this thread saw (NaN check)
  int done = 0;
  const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(r)) & 15u) == 0;
  if (vec) {
    const int nvec = len >> 2;
    const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
    float4* __restrict__ r4 = reinterpret_cast<float4*>(r);
    if (nvec == kTile / 4) {
      constexpr int U = kTile / (4 * kBlock);
      float4 a[U], b[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        a[u] = g4[u * kBlock + tid];
        b[u] = r4[u * kBlock + tid];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float4 x;
        uint32_t m;
        stream_quad(a[u], b[u], x, h, m);
        r4[u * kBlock + tid] = x;
        tmax = max(tmax, m);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        m = max(m, (uint32_t)__shfl_xor((int)m, 4));
        if ((tid & 7) == 0) lmax[(u * kBlock + tid) >> 3] = m;
      }
    } else {
      for (int base = 0; base < nvec; base += kBlock) {
        const int v = base + tid;
        uint32_t m = 0u;
        if (v < nvec) {
          float4 x;
          stream_quad(g4[v], r4[v], x, h, m);
          r4[v] = x;
          tmax = max(tmax, m);
        }
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        m = max(m, (uint32_t)__shfl_xor((int)m, 4));
        if ((tid & 7) == 0 && v < nvec) lmax[v >> 3] = m;
      }
    }
    done = nvec << 2;
  }
  __syncthreads();
  for (int e = done + tid; e < len; e += kBlock) {
    const float x = g[e] + r[e];
    r[e] = x;
    const uint32_t k = mag_key(x);
    atomicAdd(&h[k >> kH1Shift], 1u);
    atomicMax(&lmax[e / kLine], k);
    tmax = max(tmax, k);
  }
  if (tmax >= kNanKeyMin) atomicOr(&nanflag, 1u);
  __syncthreads();
  const int nlines = (len + kLine - 1) / kLine;
  if (tid < nlines) summ[t.line0 + tid] = (uint16_t)(lmax[tid] >> 16);
  uint32_t* __restrict__ gh = hist1 + (size_t)t.group * kH1Bins;
  for (int i = tid; i < kH1Bins; i += kBlock) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&gh[i], c);
  }
  if (tid == 0 && nanflag && status) atomicOr(status, TKEF_STATUS_NAN);
}

// ---------------------------------------------------------------------------
// pick: one workgroup per group. Walking the histogram from its highest bin,
// find the bin where the running count first reaches `need`.
__global__ __launch_bounds__(kBlock) void k_pick(int level, const GroupDesc* __restrict__ groups,
                                                 GroupState* __restrict__ st,
                                                 const uint32_t* __restrict__ hist, int nbins) {
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
  const uint32_t* __restrict__ hg = hist + (size_t)g * nbins;
  const int per = nbins / kBlock;
  const int hi = nbins - 1 - tid * per;
  uint32_t sum = 0u;
  for (int j = 0; j < per; ++j) sum += hg[hi - j];
  uint32_t total;
  const uint32_t excl = block_excl_scan(sum, part, &total);
  if (excl < need && need <= excl + sum) {
    uint32_t acc = excl;
    for (int j = 0; j < per; ++j) {
      const uint32_t c = hg[hi - j];
      if (acc + c >= need) {
        res[0] = (uint32_t)(hi - j);
        res[1] = acc;
        res[2] = c;
        break;
      }
      acc += c;
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
// refine: histogram of the next 10 key bits over the elements of the current
// key class (level 2: key >> 20 == prefix; level 3: key >> 10 == prefix).
__global__ __launch_bounds__(kBlock) void k_refine(int level, const TileDesc* __restrict__ tiles,
                                                   const GroupState* __restrict__ st,
                                                   const uint16_t* __restrict__ summ,
                                                   uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[kH2Bins];
  __shared__ uint32_t any;
  const int tid = threadIdx.x;
  const TileDesc t = tiles[blockIdx.x];
  const GroupState s = st[t.group];
  if (s.need == 0u) return;
  const int cshift = (level == 2) ? kH1Shift : kH2Shift;
  const int bshift = (level == 2) ? kH2Shift : 0;
  const uint32_t cls = s.prefix;
  const uint32_t sthr = (cls << cshift) >> 16;
  for (int i = tid; i < kH2Bins; i += kBlock) h[i] = 0u;
  if (tid == 0) any = 0u;
  __syncthreads();
  const int nlines = (t.len + kLine - 1) / kLine;
  if (tid < nlines && summ[t.line0 + tid] >= sthr) {
    const int e0 = tid * kLine;
    const int n = min(kLine, t.len - e0);
    float v[kLine];
    load_line(t.r, e0, n, v);
    uint32_t hit = 0u;
#pragma unroll
    for (int q = 0; q < kLine; ++q) {
      const uint32_t k = mag_key(v[q]);
      if (q < n && (k >> cshift) == cls) {
        atomicAdd(&h[(k >> bshift) & (kH2Bins - 1)], 1u);
        hit = 1u;
      }
    }
    if (hit) any = 1u;
  }
  __syncthreads();
  if (!any) return;
  uint32_t* __restrict__ gh = hist + (size_t)t.group * kH2Bins;
  for (int i = tid; i < kH2Bins; i += kBlock) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&gh[i], c);
  }
}

// ---------------------------------------------------------------------------
// count: per tile, #{key > T} (low 16 bits) and #{key == T} (high 16 bits).
__device__ __forceinline__ uint32_t line_counts(const TileDesc& t, int line, uint32_t T,
                                                const uint16_t* __restrict__ summ) {
  const int nlines = (t.len + kLine - 1) / kLine;
  if (line >= nlines || summ[t.line0 + line] < (T >> 16)) return 0u;
  const int e0 = line * kLine;
  const int n = min(kLine, t.len - e0);
  float v[kLine];
  load_line(t.r, e0, n, v);
  uint32_t gt = 0u, eq = 0u;
#pragma unroll
  for (int q = 0; q < kLine; ++q) {
    const uint32_t k = mag_key(v[q]);
    gt += (q < n && k > T) ? 1u : 0u;
    eq += (q < n && k == T) ? 1u : 0u;
  }
  return gt | (eq << 16);
}

__global__ __launch_bounds__(kBlock) void k_count(const TileDesc* __restrict__ tiles,
                                                  const GroupState* __restrict__ st,
                                                  const uint16_t* __restrict__ summ,
                                                  uint32_t* __restrict__ tile_cnt) {
  __shared__ uint32_t buf[kBlock];
  const int tid = threadIdx.x;
  const TileDesc t = tiles[blockIdx.x];
  const GroupState s = st[t.group];
  uint32_t c = (s.need == 0u) ? 0u : line_counts(t, tid, s.T, summ);
  uint32_t total;
  (void)block_excl_scan(c, buf, &total);
  if (tid == 0) {
    tile_cnt[2 * blockIdx.x + 0] = total & 0xFFFFu;
    tile_cnt[2 * blockIdx.x + 1] = total >> 16;
  }
}

// ---------------------------------------------------------------------------
// scan: one workgroup of kScanBlock threads. pre_glob = exclusive prefix of
// the per-tile (gt, eq) counts over all tiles; pre_rel = the same relative to
// the first tile of the tile's group.
constexpr int kScanBlock = 1024;

__global__ __launch_bounds__(kScanBlock) void k_scan(const TileDesc* __restrict__ tiles,
                                                     int32_t ntiles,
                                                     const GroupDesc* __restrict__ groups,
                                                     const uint32_t* __restrict__ tile_cnt,
                                                     uint32_t* __restrict__ pre_glob,
                                                     uint32_t* __restrict__ pre_rel) {
  __shared__ uint32_t sg[kScanBlock], se[kScanBlock];
  const int tid = threadIdx.x;
  const int per = (ntiles + kScanBlock - 1) / kScanBlock;
  const int b0 = min(ntiles, tid * per), b1 = min(ntiles, b0 + per);
  uint32_t lg = 0u, le = 0u;
  for (int i = b0; i < b1; ++i) {
    lg += tile_cnt[2 * i];
    le += tile_cnt[2 * i + 1];
  }
  sg[tid] = lg;
  se[tid] = le;
  __syncthreads();
  for (int off = 1; off < kScanBlock; off <<= 1) {
    const uint32_t ag = (tid >= off) ? sg[tid - off] : 0u;
    const uint32_t ae = (tid >= off) ? se[tid - off] : 0u;
    __syncthreads();
    sg[tid] += ag;
    se[tid] += ae;
    __syncthreads();
  }
  uint32_t rg = sg[tid] - lg, re = se[tid] - le;
  for (int i = b0; i < b1; ++i) {
    pre_glob[2 * i] = rg;
    pre_glob[2 * i + 1] = re;
    rg += tile_cnt[2 * i];
    re += tile_cnt[2 * i + 1];
  }
  __syncthreads();
  for (int i = b0; i < b1; ++i) {
    const uint32_t first = groups[tiles[i].group].tile_begin;
    pre_rel[2 * i] = pre_glob[2 * i] - pre_glob[2 * first];
    pre_rel[2 * i + 1] = pre_glob[2 * i + 1] - pre_glob[2 * first + 1];
  }
}

// ---------------------------------------------------------------------------
// emit: ordered compaction. An element with key > T goes to slot
// (#gt before it) + min(#eq before it, need); an element with key == T is
// kept while fewer than `need` equal keys precede it in its group.
__global__ __launch_bounds__(kBlock) void k_emit(const TileDesc* __restrict__ tiles,
                                                 const GroupDesc* __restrict__ groups,
                                                 const GroupState* __restrict__ st,
                                                 const uint16_t* __restrict__ summ,
                                                 const uint32_t* __restrict__ pre_rel,
                                                 int32_t* __restrict__ idx_out,
                                                 float* __restrict__ val_out) {
  __shared__ uint32_t buf[kBlock];
  const int tid = threadIdx.x;
  const TileDesc t = tiles[blockIdx.x];
  const GroupState s = st[t.group];
  if (s.need == 0u) return;
  const GroupDesc gd = groups[t.group];
  const uint32_t T = s.T, need = s.need;
  const int nlines = (t.len + kLine - 1) / kLine;
  const bool flagged = tid < nlines && summ[t.line0 + tid] >= (T >> 16);
  const int e0 = tid * kLine;
  const int n = flagged ? min(kLine, t.len - e0) : 0;
  float v[kLine];
  uint32_t c = 0u;
  if (flagged) {
    load_line(t.r, e0, n, v);
    uint32_t gt = 0u, eq = 0u;
#pragma unroll
    for (int q = 0; q < kLine; ++q) {
      const uint32_t k = mag_key(v[q]);
      gt += (q < n && k > T) ? 1u : 0u;
      eq += (q < n && k == T) ? 1u : 0u;
    }
    c = gt | (eq << 16);
  }
  uint32_t total;
  const uint32_t ex = block_excl_scan(c, buf, &total);
  if (c == 0u) return;
  uint32_t gtr = pre_rel[2 * blockIdx.x] + (ex & 0xFFFFu);
  uint32_t eqr = pre_rel[2 * blockIdx.x + 1] + (ex >> 16);
  float* __restrict__ r = t.r;
#pragma unroll
  for (int q = 0; q < kLine; ++q) {
    if (q >= n) break;
    const uint32_t k = mag_key(v[q]);
    uint32_t pos = 0xFFFFFFFFu;
    if (k > T) {
      pos = gtr + min(eqr, need);
      ++gtr;
    } else if (k == T) {
      if (eqr < need) pos = gtr + eqr;
      ++eqr;
    }
    if (pos < gd.k) {
      idx_out[gd.out_base + pos] = t.gstart + e0 + q;
      val_out[gd.out_base + pos] = v[q];
      r[e0 + q] = 0.0f;
    }
  }
}

// ---------------------------------------------------------------------------
// seg: seg[p][u] = first entry of worker p's list whose index lies in update
// tile u or later; seg[p][ntiles_u] = nnz_p. Also flags unsorted or
// out-of-range lists in the status word.
__global__ void k_seg(const int32_t* __restrict__ idx, int64_t stride,
                      const int32_t* __restrict__ nnz, int32_t d, int32_t ntiles_u,
                      int32_t* __restrict__ seg, uint32_t* __restrict__ status) {
  const int p = blockIdx.y;
  int64_t n = nnz ? (int64_t)nnz[p] : stride;
  n = n < 0 ? 0 : (n > stride ? stride : n);
  const int32_t* __restrict__ L = idx + (int64_t)p * stride;
  int32_t* __restrict__ S = seg + (int64_t)p * (ntiles_u + 1);
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n == 0) {
    for (int64_t u = j; u <= ntiles_u; u += (int64_t)gridDim.x * blockDim.x) S[u] = 0;
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
  for (int32_t u = tp + 1; u <= t; ++u) S[u] = (int32_t)j;
  if (j == n - 1)
    for (int32_t u = t + 1; u <= ntiles_u; ++u) S[u] = (int32_t)n;
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

__global__ __launch_bounds__(kUBlock) void k_update(
    const UpdTensor* __restrict__ tens, const int32_t* __restrict__ tile_first, int32_t ntens,
    int32_t d, int32_t ntiles_u, const int32_t* __restrict__ idx, const float* __restrict__ val,
    int64_t stride, const int32_t* __restrict__ nnz, int32_t P, const int32_t* __restrict__ seg,
    float lr, float mu, float wd, int sparse_mode, int has_mom) {
  __shared__ float acc[kUTile];
  __shared__ uint32_t mask[kUTile / 32];
  __shared__ int32_t sbeg[kUBlock];
  __shared__ uint32_t scan[kUBlock];
  const int tid = threadIdx.x;
  const int u = blockIdx.x;
  const int32_t base = u << kUShift;
  const int32_t len = min(kUTile, d - base);
  for (int i = tid; i < kUTile; i += kUBlock) acc[i] = 0.0f;
  for (int i = tid; i < kUTile / 32; i += kUBlock) mask[i] = 0u;
  __syncthreads();

  // 1. accumulate every worker's entries that fall in this tile
  for (int p0 = 0; p0 < P; p0 += kUBlock) {
    const int p = p0 + tid;
    int32_t b = 0, e = 0;
    if (p < P) {
      int64_t np = nnz ? (int64_t)nnz[p] : stride;
      np = np < 0 ? 0 : (np > stride ? stride : np);
      const int32_t* S = seg + (int64_t)p * (ntiles_u + 1);
      int64_t sb = S[u], se = S[u + 1];
      sb = sb < 0 ? 0 : (sb > np ? np : sb);
      se = se < sb ? sb : (se > np ? np : se);
      b = (int32_t)sb;
      e = (int32_t)se;
    }
    sbeg[tid] = b;
    uint32_t total;
    const uint32_t ex = block_excl_scan((uint32_t)(e - b), scan, &total);
    scan[tid] = ex + (uint32_t)(e - b);  // inclusive, read after the barrier
    __syncthreads();
    for (uint32_t q = tid; q < total; q += kUBlock) {
      int lo = 0, hi = kUBlock - 1;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (scan[mid] > q) hi = mid; else lo = mid + 1;
      }
      const uint32_t before = lo ? scan[lo - 1] : 0u;
      const int64_t gi = (int64_t)(p0 + lo) * stride + sbeg[lo] + (q - before);
      const int32_t li = idx[gi] - base;
      if (li >= 0 && li < len) {
        atomicAdd(&acc[li], val[gi]);
        if (sparse_mode) atomicOr(&mask[li >> 5], 1u << (li & 31));
      }
    }
    __syncthreads();
  }

  // 2. apply the SGD step
  const int32_t t0 = tile_first[u];
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
    const bool mom = has_mom != 0;
    float* __restrict__ bm = mom ? tt.b + (a - tt.goff) : nullptr;
    const bool vec = ((reinterpret_cast<uintptr_t>(w) |
                       (bm ? reinterpret_cast<uintptr_t>(bm) : 0u)) & 15u) == 0;
    int done = 0;
    if (vec) {
      const int nv = cnt >> 2;
      float4* w4 = reinterpret_cast<float4*>(w);
      float4* b4 = reinterpret_cast<float4*>(bm);
      for (int q = tid; q < nv; q += kUBlock) {
        float4 wv = w4[q];
        float4 bv = bm ? b4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
        const int l = la + 4 * q;
        float b0 = bv.x, b1 = bv.y, b2 = bv.z, b3 = bv.w;
        wv.x = sgd_step(acc[l + 0], wv.x, b0, mom, lr, mu, wd);
        wv.y = sgd_step(acc[l + 1], wv.y, b1, mom, lr, mu, wd);
        wv.z = sgd_step(acc[l + 2], wv.z, b2, mom, lr, mu, wd);
        wv.w = sgd_step(acc[l + 3], wv.w, b3, mom, lr, mu, wd);
        w4[q] = wv;
        if (mom) b4[q] = make_float4(b0, b1, b2, b3);
      }
      done = nv << 2;
    }
    for (int q = done + tid; q < cnt; q += kUBlock) {
      float bv = mom ? bm[q] : 0.0f;
      w[q] = sgd_step(acc[la + q], w[q], bv, mom, lr, mu, wd);
      if (mom) bm[q] = bv;
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

hipError_t launch_stream(const TileDesc* tiles, int32_t ntiles, uint32_t* hist1,
                         uint16_t* summ, uint32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(k_stream, dim3(ntiles), dim3(kBlock), 0, s, tiles, hist1, summ, status);
  return hipGetLastError();
}

hipError_t launch_pick(int level, const GroupDesc* groups, GroupState* st,
                       const uint32_t* hist, int32_t ngroups, hipStream_t s) {
  const int nbins = (level == 1) ? kH1Bins : kH2Bins;
  hipLaunchKernelGGL(k_pick, dim3(ngroups), dim3(kBlock), 0, s, level, groups, st, hist, nbins);
  return hipGetLastError();
}

hipError_t launch_refine(int level, const TileDesc* tiles, int32_t ntiles,
                         const GroupState* st, const uint16_t* summ, uint32_t* hist,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_refine, dim3(ntiles), dim3(kBlock), 0, s, level, tiles, st, summ, hist);
  return hipGetLastError();
}

hipError_t launch_count(const TileDesc* tiles, int32_t ntiles, const GroupState* st,
                        const uint16_t* summ, uint32_t* tile_cnt, hipStream_t s) {
  hipLaunchKernelGGL(k_count, dim3(ntiles), dim3(kBlock), 0, s, tiles, st, summ, tile_cnt);
  return hipGetLastError();
}

hipError_t launch_scan(const TileDesc* tiles, int32_t ntiles, const GroupDesc* groups,
                       const uint32_t* tile_cnt, uint32_t* pre_glob, uint32_t* pre_rel,
                       hipStream_t s) {
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, s, tiles, ntiles, groups, tile_cnt,
                     pre_glob, pre_rel);
  return hipGetLastError();
}

hipError_t launch_emit(const TileDesc* tiles, int32_t ntiles, const GroupDesc* groups,
                       const GroupState* st, const uint16_t* summ, const uint32_t* pre_rel,
                       int32_t* idx_out, float* val_out, hipStream_t s) {
  hipLaunchKernelGGL(k_emit, dim3(ntiles), dim3(kBlock), 0, s, tiles, groups, st, summ, pre_rel,
                     idx_out, val_out);
  return hipGetLastError();
}

hipError_t launch_seg(const int32_t* idx, int64_t stride, const int32_t* nnz, int32_t P,
                      int32_t d, int32_t ntiles_u, int32_t* seg, uint32_t* status,
                      hipStream_t s) {
  int64_t bx = (stride + 255) / 256;
  if (bx < 1) bx = 1;
  hipLaunchKernelGGL(k_seg, dim3((unsigned)bx, (unsigned)P), dim3(256), 0, s, idx, stride, nnz,
                     d, ntiles_u, seg, status);
  return hipGetLastError();
}

hipError_t launch_update(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                         int32_t d, int32_t ntiles_u, const int32_t* idx, const float* val,
                         int64_t stride, const int32_t* nnz, int32_t P, const int32_t* seg,
                         float lr, float mu, float wd, int sparse_mode, int has_mom,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_update, dim3(ntiles_u), dim3(kUBlock), 0, s, tens, tile_first, ntens, d,
                     ntiles_u, idx, val, stride, nnz, P, seg, lr, mu, wd, sparse_mode, has_mom);
  return hipGetLastError();
}

}  // namespace tkef

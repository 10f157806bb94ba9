// Host side of the tkef C ABI: argument validation, plans, workspace layout
// and the launch sequence. No device memory is allocated here; every device
// buffer is the caller's.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include <hip/hip_runtime_api.h>

#include "tkef.h"
#include "tkef_internal.h"

using namespace tkef;

namespace {

constexpr int64_t kMaxD = 2147483647LL;  // positions are int32
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

bool aligned_ws(const void* ws) {
  return (reinterpret_cast<uintptr_t>(ws) & (kAlign - 1)) == 0;
}

int hip_rc(hipError_t e) { return e == hipSuccess ? TKEF_OK : TKEF_EHIP; }

bool ranges_overlap(const void* a, const void* b, int64_t n) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  const uintptr_t bytes = static_cast<uintptr_t>(n) * sizeof(float);
  return x < y + bytes && y < x + bytes;
}

// Validates a tensor-size list: sizes >= 0, total in [1, kMaxD].
int check_numels(const int64_t* numels, int32_t ntensors, int64_t* total) {
  if (!numels || ntensors <= 0) return TKEF_EINVAL;
  int64_t d = 0;
  for (int32_t t = 0; t < ntensors; ++t) {
    if (numels[t] < 0) return TKEF_EINVAL;
    if (numels[t] > kMaxD) return TKEF_ERANGE;
    d += numels[t];
    if (d > kMaxD) return TKEF_ERANGE;
  }
  if (d < 1) return TKEF_ERANGE;
  *total = d;
  return TKEF_OK;
}

// Optional timing events of an execution: ev[0] is recorded at the start of
// launch 0 and ev[i + 1] at the end of launch i, by the dispatches themselves
// (no separate event commands between the kernels).
struct Tracer {
  hipEvent_t* ev;
  int32_t n;
  Ev at(int i) const {
    Ev e;
    if (!ev) return e;
    if (i == 0 && n > 0) e.start = ev[0];
    if (i + 1 < n) e.stop = ev[i + 1];
    return e;
  }
};

}  // namespace

// ============================================================================
// shared helpers

extern "C" int tkef_version(void) { return TKEF_VERSION; }

extern "C" const char* tkef_strerror(int code) {
  switch (code) {
    case TKEF_OK: return "ok";
    case TKEF_EINVAL: return "invalid argument (null pointer, bad mode or count, aliasing)";
    case TKEF_ERANGE: return "out of range (size >= 2^31, k outside [1, d], rho outside (0, 1])";
    case TKEF_EWORKSPACE: return "workspace missing, too small or not 256-byte aligned";
    case TKEF_EHIP: return "HIP runtime error";
    case TKEF_ESTATE: return "plan not bound, or bound to a different workspace";
    case TKEF_ENOMEM: return "host allocation failed";
    default: return "unknown tkef error code";
  }
}

extern "C" int64_t tkef_k_from_rho(int64_t d, double rho) {
  if (d < 0 || !(rho > 0.0 && rho <= 1.0) || !std::isfinite(rho)) return TKEF_ERANGE;
  if (d == 0) return 0;
  const double kd = std::ceil(rho * static_cast<double>(d));
  // clamped in double first: rho * d can round up to 2^63, which int64_t
  // cannot hold
  if (kd >= static_cast<double>(d)) return d;
  int64_t k = static_cast<int64_t>(kd);
  if (k < 1) k = 1;
  if (k > d) k = d;
  return k;
}

// ============================================================================
// sparsify plan

// Launch sequences: one selection group (global) and several (per tensor).
static const char* const kSparsifyLaunchesOne[] = {"stream", "collect", "finish"};
static const char* const kSparsifyLaunchesMany[] = {"stream", "pick1", "gather",
                                                    "pick2",  "hist3", "pick3",
                                                    "groupscan", "emit"};
// up to emit_lds_groups() groups, emit forms the group bases itself
static const char* const kSparsifyLaunchesFold[] = {"stream", "pick1", "gather", "pick2",
                                                    "hist3",  "pick3", "emit"};
constexpr int32_t kSparsifyNLaunchOne = 3, kSparsifyNLaunchMany = 8, kSparsifyNLaunchFold = 7;
// MSTopK: stream, count, refine x (passes - 1), emit
static const char* const kApproxRefine[] = {"ms_refine1", "ms_refine2", "ms_refine3",
                                            "ms_refine4", "ms_refine5", "ms_refine6",
                                            "ms_refine7"};
// passes for n rounds: six in the first, twelve in each later one
constexpr int32_t ms_passes_for(int32_t n) {
  return 1 + (n > kMsRoundsPerPass
                  ? (n - kMsRoundsPerPass + kMsRoundsPerRefine - 1) / kMsRoundsPerRefine
                  : 0);
}
constexpr int32_t kMsMaxPasses = ms_passes_for(kMsMaxRounds);
static_assert(kMsMaxPasses - 1 <= 7, "refine names");
// counters of the first pass (kMsSlots copies of 64), then one copy of
// kMsRefineBins per later pass
constexpr size_t kMsCntWords =
    (size_t)kMsSlots * 64 + (size_t)(kMsMaxPasses - 1) * kMsRefineBins;

struct tkef_sparsify_plan_s {
  int32_t ntensors = 0, mode = 0, ngroups = 0, ntiles = 0, nslots = 1, stream_grid = 1;
  int32_t count_grid = 1;  // MSTopK first counting pass: eight workgroups per compute unit
  // per-tensor path: gather runs one workgroup per line region (line_grid),
  // hist3 and emit split the candidates over cand_grid workgroups (at least
  // line_grid, which their line walk after an overflow needs; at most
  // sel_grid, which sizes their flag arrays)
  int32_t line_grid = 1, cand_grid = 1;
  int64_t d = 0, k_total = 0, nlines = 0;
  std::vector<int64_t> numels, goff, kgroup;
  std::vector<TileDesc> tiles;   // pointers filled at bind
  std::vector<GroupDesc> groups;
  uint32_t cand_cap = 0;  // per-tensor path: capacity of the compacted candidate list
  uint32_t rcap = 0;      // one-group path: candidates stored per region
  int32_t sel_lpt = 1, sel_grid = 1, sel_block = 1;  // selection kernels: lines per thread,
                                                    // workgroups, threads per workgroup
  // Scratch that must start at zero (histograms, prefix flags, overflow and
  // count words), at off_zero; offsets below are relative to it. It is laid
  // out so that what the execution's last kernel uses comes last, from
  // zero_tail on: the first kernel (the stream) clears that part, which it
  // does not use, and the last kernel clears the part before zero_tail,
  // which only earlier kernels use. Every execution thus launches the same
  // kernels with the same arguments (a captured execution can be replayed).
  size_t off_tiles = 0, off_groups = 0, off_state = 0, off_zero = 0, zero_bytes = 0,
         zero_tail = 0,
         off_hist1 = 0, off_hist2 = 0, off_hist3 = 0, off_flags1 = 0, off_flags2 = 0,
         off_meta = 0, off_summ = 0, off_base = 0, off_cand = 0, off_rcand = 0, off_rband = 0,
         off_rsuf = 0, off_rcnt = 0, off_rbin = 0, off_rbtmp = 0, off_ticket = 0, off_rzr = 0,
         ws_bytes = 0;
  int32_t val_format = TKEF_VAL_F32;  // value array written by execute
  // MSTopK (TKEF_APPROX): rounds, offset word, scratch
  int32_t ms_rounds = 30;
  uint64_t ms_word = 0;
  size_t off_ms_state = 0, off_ms_esum = 0, off_ms_emax = 0, off_ms_cnt = 0,
         off_ms_flags = 0;  // state: kMsMaxPasses + 1 records, zeroed scratch: the rest
  bool needs_clear = true;   // the zeroed scratch must be cleared before the next run
  int32_t ms_passes() const { return ms_passes_for(ms_rounds); }
  int32_t nlaunch() const {
    if (mode == TKEF_APPROX) return 2 + ms_passes();
    if (ngroups == 1) return kSparsifyNLaunchOne;
    return ngroups <= emit_lds_groups() ? kSparsifyNLaunchFold : kSparsifyNLaunchMany;
  }
  void* bound_ws = nullptr;
  hipEvent_t* events = nullptr;
  int32_t n_events = 0;
};

// Launch shapes and workspace layout of a sparsify plan from its sizes (mode,
// d, ngroups, k_total, ntiles, nlines); allocates nothing. False when the
// selection grids cannot cover the tiles.
bool sparsify_layout(tkef_sparsify_plan_s* p) {
  // selection kernels: `lpt` consecutive summary lines per thread, at most
  // select_max_groups() workgroups of sb threads (collect_block() for the
  // exact one-group kernels, select_block() for the others). Aim for about
  // 256 workgroups (one per compute unit); lpt is a power of two from 4 up
  // (the kernels fetch four 16-bit summaries per load, and a thread's lines
  // must lie in one tile).
  const bool one = p->ngroups == 1;
  const bool approx = p->mode == TKEF_APPROX;
  const bool coll = one && !approx;
  const int64_t sb = coll ? collect_block(p->nlines, p->k_total, p->d) : select_block();
  p->sel_block = (int32_t)sb;
  const int64_t sg = select_max_groups();
  const int64_t want = (p->nlines + sb * 256 - 1) / (sb * 256);
  int64_t lpt = 4;  // a power of two from 4 to select_max_lpt()
  while (lpt < want && lpt < select_max_lpt()) lpt *= 2;
  if ((p->nlines + sb * lpt - 1) / (sb * lpt) > sg) return false;  // (kMaxTiles)
  p->sel_lpt = (int32_t)lpt;
  const int64_t g_lines = (p->nlines + sb * lpt - 1) / (sb * lpt);
  // Candidates are the positions at or above the level-1 threshold bin:
  // about k plus one bin's worth. One group: each region (the lines of one
  // workgroup) stores up to rcap of them, several times the even share of
  // 8k + 65536, and at least 1/64 of the region (a level-1 bin, 1/8 of an
  // octave, can hold a percent of the data when the residual has piled mass
  // just below the threshold); per tensor: one compacted list of
  // 4k + 65536. Heavier inputs fall back to re-reading lines.
  if (one) {
    p->sel_grid = (int32_t)std::max<int64_t>(1, g_lines);
    const int64_t region = lpt * sb * kLine;
    const int64_t share = (8 * p->k_total + 65536 + p->sel_grid - 1) / p->sel_grid;
    p->rcap = (uint32_t)std::min<int64_t>(
        region, std::max<int64_t>(std::max<int64_t>(4096, (share + 63) / 64 * 64), region / 64));
  } else {
    p->cand_cap = (uint32_t)std::min<int64_t>(p->d, 4 * p->k_total + 65536);
    const int64_t g_cands = std::min<int64_t>(sg, ((int64_t)p->cand_cap + sb * 4 - 1) / (sb * 4));
    p->sel_grid = (int32_t)std::max<int64_t>(1, std::max(g_lines, g_cands));
    p->line_grid = (int32_t)std::max<int64_t>(1, g_lines);
  }
  // level-1 histogram copies per group: many for one global selection (all
  // workgroups add into it), a few per tensor in per-tensor mode
  p->nslots = one ? kSlotsOne : kSlotsMany;

  // workspace layout (every region 256-B aligned)
  size_t o = 0;
  p->off_tiles = o;   o = align_up(o + (size_t)p->ntiles * sizeof(TileDesc));
  p->off_groups = o;  o = align_up(o + (size_t)p->ngroups * sizeof(GroupDesc));
  p->off_state = o;   o = align_up(o + (size_t)p->ngroups * sizeof(GroupState));
  size_t z = 0;
  if (approx) {
    p->off_ms_state = o;  o = align_up(o + (size_t)(kMsMaxPasses + 1) * sizeof(MsState));
    p->off_ms_esum = z;   z = align_up(z + (size_t)kMsSlots * kMsDigitStride * 8);
    p->off_ms_emax = z;   z = align_up(z + (size_t)kMsSlots * 4);
    p->off_ms_cnt = z;    z = align_up(z + kMsCntWords * 4);
    p->off_ms_flags = z;  z = align_up(z + (size_t)p->sel_grid * 8);
  } else {
    p->off_hist1 = z;   z = align_up(z + (size_t)p->ngroups * p->nslots * kH1Bins * 4);
    p->off_hist2 = z;   z = align_up(z + (size_t)p->ngroups * kH2Bins * 4);
    if (one) {
      p->off_ticket = z;  z = align_up(z + 4);  // finish's last-workgroup ticket
    }
  }
  if (!one) {
    p->off_hist3 = z;   z = align_up(z + (size_t)p->ngroups * kH3Bins * 4);
    p->off_flags1 = z;  z = align_up(z + (size_t)p->sel_grid * 8);
    p->off_flags2 = z;  z = align_up(z + (size_t)p->sel_grid * 8);
    p->off_meta = z;    z = align_up(z + 8);
  }
  p->zero_bytes = z;
  // the last kernel's part: finish uses hist2 and its ticket; emit the second
  // prefix flags and meta; MSTopK's emit the last pass's counts and its flags
  // (that start depends on the rounds: see zero_split)
  p->zero_tail = approx ? p->off_ms_cnt : (one ? p->off_hist2 : p->off_flags2);
  p->off_zero = o;    o = align_up(o + z);
  p->off_summ = o;    o = align_up(o + (size_t)p->nlines * sizeof(uint16_t));
  if (approx) {
    // no candidate tables: the passes read the lines again
  } else if (one) {
    const size_t slots = (size_t)p->sel_grid * p->rcap;
    p->off_rcand = o;  o = align_up(o + slots * 16);
    p->off_rband = o;  o = align_up(o + slots * 4);
    p->off_rbtmp = o;  o = align_up(o + slots * 4);
    p->off_rsuf = o;   o = align_up(o + (size_t)p->sel_grid * kH2Bins * 4);
    p->off_rcnt = o;   o = align_up(o + (size_t)p->sel_grid * 8);
    p->off_rbin = o;   o = align_up(o + (size_t)kH2Bins * p->sel_grid * kPerBin * 4);
    p->off_rzr = o;    o = align_up(o + (size_t)p->sel_grid * 8);  // deferred residual slots
  } else {
    p->off_base = o;   o = align_up(o + (size_t)p->ngroups * 8);
    p->off_cand = o;   o = align_up(o + (size_t)p->cand_cap * 8);  // {code, bits of x}
  }
  p->ws_bytes = o;
  return true;
}

extern "C" int tkef_sparsify_plan_create(const int64_t* numels, int32_t ntensors, int32_t mode,
                                         double rho, int64_t k, tkef_sparsify_plan* plan_out) {
  if (!plan_out) return TKEF_EINVAL;
  *plan_out = nullptr;
  int64_t d = 0;
  int rc = check_numels(numels, ntensors, &d);
  if (rc) return rc;
  if (mode != TKEF_GLOBAL && mode != TKEF_PER_TENSOR && mode != TKEF_APPROX) return TKEF_EINVAL;
  if (k < 0) return TKEF_ERANGE;
  if (k > 0) {
    if (mode == TKEF_PER_TENSOR) return TKEF_EINVAL;
    if (k > d) return TKEF_ERANGE;
  } else if (!(rho > 0.0 && rho <= 1.0) || !std::isfinite(rho)) {
    return TKEF_ERANGE;
  }
  int64_t ntiles = 0;
  for (int32_t t = 0; t < ntensors; ++t) ntiles += (numels[t] + kTile - 1) / kTile;
  if (ntiles > kMaxTiles) return TKEF_ERANGE;
  tkef_sparsify_plan p = new (std::nothrow) tkef_sparsify_plan_s();
  if (!p) return TKEF_ENOMEM;
  try {
    p->ntensors = ntensors;
    p->mode = mode;
    p->d = d;
    p->numels.assign(numels, numels + ntensors);
    p->goff.resize(ntensors);
    int64_t off = 0;
    for (int32_t t = 0; t < ntensors; ++t) {
      p->goff[t] = off;
      off += numels[t];
    }
    p->ngroups = (mode == TKEF_PER_TENSOR) ? ntensors : 1;
    p->kgroup.assign(p->ngroups, 0);
    if (mode != TKEF_PER_TENSOR) {
      p->kgroup[0] = (k > 0) ? k : tkef_k_from_rho(d, rho);
    } else {
      for (int32_t t = 0; t < ntensors; ++t) p->kgroup[t] = tkef_k_from_rho(numels[t], rho);
    }
    p->k_total = 0;
    for (int64_t kg : p->kgroup) p->k_total += kg;

    // tiles: tensor-major, kTile elements each
    p->groups.assign(p->ngroups, GroupDesc{0, 0, 0, 0});
    int64_t out = 0;
    for (int32_t t = 0; t < ntensors; ++t) {
      const int32_t grp = (mode == TKEF_PER_TENSOR) ? t : 0;
      if (mode == TKEF_PER_TENSOR || t == 0) {
        p->groups[grp].k = static_cast<uint32_t>(p->kgroup[grp]);
        p->groups[grp].tile_begin = static_cast<uint32_t>(p->tiles.size());
        p->groups[grp].out_base = static_cast<uint32_t>(out);
        out += p->kgroup[grp];
      }
      for (int64_t s = 0; s < numels[t]; s += kTile) {
        TileDesc td;
        td.g = nullptr;
        td.r = nullptr;
        td.gstart = static_cast<int32_t>(p->goff[t] + s);
        td.len = static_cast<int32_t>(std::min<int64_t>(kTile, numels[t] - s));
        td.group = grp;
        td.reserved = 0;
        p->tiles.push_back(td);
      }
    }
    p->ntiles = static_cast<int32_t>(p->tiles.size());
    p->nlines = (int64_t)p->ntiles * kLinesPerTile;
    if (!sparsify_layout(p)) throw std::bad_alloc();  // (excluded by kMaxTiles above)
  } catch (const std::bad_alloc&) {
    delete p;
    return TKEF_ENOMEM;
  }
  *plan_out = p;
  return TKEF_OK;
}

extern "C" int tkef_sparsify_plan_destroy(tkef_sparsify_plan plan) {
  delete plan;
  return TKEF_OK;
}

extern "C" int tkef_sparsify_plan_info(tkef_sparsify_plan plan, size_t* workspace_bytes,
                                       int64_t* k_total, int64_t* d_total, int32_t* ngroups,
                                       int32_t* nlaunch) {
  if (!plan) return TKEF_EINVAL;
  if (workspace_bytes) *workspace_bytes = plan->ws_bytes;
  if (k_total) *k_total = plan->k_total;
  if (d_total) *d_total = plan->d;
  if (ngroups) *ngroups = plan->ngroups;
  if (nlaunch) *nlaunch = plan->nlaunch();
  return TKEF_OK;
}

extern "C" int tkef_sparsify_plan_group_k(tkef_sparsify_plan plan, int64_t* k_out, int32_t n) {
  if (!plan || !k_out || n < plan->ngroups) return TKEF_EINVAL;
  for (int32_t g = 0; g < plan->ngroups; ++g) k_out[g] = plan->kgroup[g];
  return TKEF_OK;
}

namespace {

// The exact selection of one group: stream, collect, finish. The workspace at
// base is laid out by sparsify_layout, its tables are written and the zeroed
// scratch starts at zb. The stream clears stream_words words at
// stream_clear, finish clear_words words at clear_next (the two parts of the
// zeroed scratch; none for a caller that clears it all beforehand).
hipError_t run_one_group(const tkef_sparsify_plan_s* p, char* base, char* zb,
                         uint32_t* stream_clear, int64_t stream_words, uint32_t* clear_next,
                         int64_t clear_words, int32_t* idx_out, void* val_out, int val16,
                         uint32_t* status, hipStream_t s, const Tracer& tr) {
  const TileDesc* tiles = reinterpret_cast<const TileDesc*>(base + p->off_tiles);
  const GroupDesc* groups = reinterpret_cast<const GroupDesc*>(base + p->off_groups);
  GroupState* st = reinterpret_cast<GroupState*>(base + p->off_state);
  uint32_t* hist1 = reinterpret_cast<uint32_t*>(zb + p->off_hist1);
  uint32_t* hist2 = reinterpret_cast<uint32_t*>(zb + p->off_hist2);
  uint16_t* summ = reinterpret_cast<uint16_t*>(base + p->off_summ);
  uint32_t* rcand = reinterpret_cast<uint32_t*>(base + p->off_rcand);
  uint32_t* rband = reinterpret_cast<uint32_t*>(base + p->off_rband);
  uint32_t* rbtmp = reinterpret_cast<uint32_t*>(base + p->off_rbtmp);
  uint32_t* rsuf = reinterpret_cast<uint32_t*>(base + p->off_rsuf);
  uint32_t* rcnt = reinterpret_cast<uint32_t*>(base + p->off_rcnt);
  uint32_t* rbin = reinterpret_cast<uint32_t*>(base + p->off_rbin);
  const int64_t nl = p->nlines;
  const int lpt = p->sel_lpt, sg = p->sel_grid;
  hipError_t e = launch_stream(tiles, p->ntiles, p->stream_grid, hist1, p->nslots, summ, status,
                               stream_clear, stream_words, s, tr.at(0));
  if (e == hipSuccess)
    e = launch_collect(tiles, groups, st, hist1, p->nslots, summ, nl, lpt, sg, p->sel_block,
                       p->rcap, hist2, rbin, rcand, rband, rbtmp, rsuf, rcnt, s, tr.at(1));
  if (e == hipSuccess)
    e = launch_finish(tiles, groups, st, summ, nl, lpt, sg, p->sel_block, p->rcap, hist2, rbin,
                      rcand, rband, rsuf, rcnt, idx_out, val_out, val16, clear_next, clear_words,
                      reinterpret_cast<uint32_t*>(zb + p->off_ticket),
                      reinterpret_cast<uint32_t*>(base + p->off_rzr), s, tr.at(2));
  return e;
}

// Persistent stream grid: four workgroups per compute unit.
int stream_grid_for(int64_t ntiles, int32_t* grid, int32_t* cus_out) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return TKEF_EHIP;
  const int64_t units = ntiles * (kTile / kStreamUnit);
  *grid = (int32_t)std::min<int64_t>((int64_t)4 * cus, units);
  if (cus_out) *cus_out = cus;
  return TKEF_OK;
}

}  // namespace

extern "C" int tkef_sparsify_plan_bind(tkef_sparsify_plan plan, const float* const* grads,
                                       float* const* residuals, void* ws, size_t ws_bytes,
                                       hipStream_t stream) {
  if (!plan || !grads || !residuals) return TKEF_EINVAL;
  if (!ws || !aligned_ws(ws) || ws_bytes < plan->ws_bytes) return TKEF_EWORKSPACE;
  for (int32_t t = 0; t < plan->ntensors; ++t) {
    const int64_t n = plan->numels[t];
    if (n == 0) continue;
    if (!grads[t] || !residuals[t]) return TKEF_EINVAL;
    if (ranges_overlap(grads[t], residuals[t], n)) return TKEF_EINVAL;
  }
  size_t i = 0;
  for (int32_t t = 0; t < plan->ntensors; ++t) {
    for (int64_t s = 0; s < plan->numels[t]; s += kTile, ++i) {
      plan->tiles[i].g = grads[t] + s;
      plan->tiles[i].r = residuals[t] + s;
    }
  }
  int32_t cus = 0;
  if (stream_grid_for(plan->ntiles, &plan->stream_grid, &cus)) return TKEF_EHIP;
  const int64_t units = (int64_t)plan->ntiles * (kTile / kStreamUnit);
  plan->count_grid = (int32_t)std::max<int64_t>(1, std::min<int64_t>((int64_t)8 * cus, (units + 1) / 2));
  // two candidate workgroups per compute unit are all resident at once
  plan->cand_grid = std::max(plan->line_grid, std::min(plan->sel_grid, 2 * cus));
  char* base = static_cast<char*>(ws);
  hipError_t e = hipMemcpyAsync(base + plan->off_tiles, plan->tiles.data(),
                                plan->tiles.size() * sizeof(TileDesc), hipMemcpyHostToDevice,
                                stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(base + plan->off_groups, plan->groups.data(),
                       plan->groups.size() * sizeof(GroupDesc), hipMemcpyHostToDevice, stream);
  // the zero-initialised scratch starts cleared
  if (e == hipSuccess)
    e = launch_fill_u32(reinterpret_cast<uint32_t*>(base + plan->off_zero), 0u,
                        (int64_t)(plan->zero_bytes / 4), stream);
  // line summaries start at 0: the stream rewrites those of lines holding
  // elements on every run and never writes the others
  if (e == hipSuccess)
    e = launch_fill_u32(reinterpret_cast<uint32_t*>(base + plan->off_summ), 0u,
                        (int64_t)(plan->nlines * sizeof(uint16_t) / 4), stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    plan->bound_ws = nullptr;
    return TKEF_EHIP;
  }
  plan->bound_ws = ws;
  plan->needs_clear = false;
  return TKEF_OK;
}

extern "C" int tkef_sparsify_plan_set_events(tkef_sparsify_plan plan, hipEvent_t* events,
                                             int32_t n_events) {
  if (!plan || n_events < 0 || (events && n_events == 0)) return TKEF_EINVAL;
  plan->events = events;
  plan->n_events = events ? n_events : 0;
  return TKEF_OK;
}

extern "C" const char* tkef_sparsify_plan_launch_name(tkef_sparsify_plan plan, int32_t i) {
  if (!plan || i < 0 || i >= plan->nlaunch()) return nullptr;
  if (plan->mode == TKEF_APPROX) {
    if (i == 0) return "ms_stream";
    if (i == 1) return "ms_count";
    if (i == plan->nlaunch() - 1) return "ms_emit";
    return kApproxRefine[i - 2];
  }
  if (plan->ngroups == 1) return kSparsifyLaunchesOne[i];
  return plan->ngroups <= emit_lds_groups() ? kSparsifyLaunchesFold[i] : kSparsifyLaunchesMany[i];
}

extern "C" int tkef_sparsify_plan_set_approx(tkef_sparsify_plan plan, int32_t n_search,
                                             uint64_t window_word) {
  if (!plan || plan->mode != TKEF_APPROX || n_search < 1 || n_search > kMsMaxRounds)
    return TKEF_EINVAL;
  plan->ms_rounds = n_search;
  plan->ms_word = window_word;
  return TKEF_OK;
}

extern "C" int tkef_sparsify_plan_set_value_format(tkef_sparsify_plan plan, int32_t format) {
  if (!plan || (format != TKEF_VAL_F32 && format != TKEF_VAL_F16)) return TKEF_EINVAL;
  plan->val_format = format;
  return TKEF_OK;
}

extern "C" int tkef_sparsify_approx_result(tkef_sparsify_plan plan, void* ws, double* out,
                                           int64_t* cnt, hipStream_t s) {
  if (!plan || plan->mode != TKEF_APPROX) return TKEF_EINVAL;
  if (!ws || plan->bound_ws != ws) return TKEF_ESTATE;
  MsState h;
  const char* base = static_cast<const char*>(ws);
  const size_t fin = plan->off_ms_state + (size_t)plan->ms_passes() * sizeof(MsState);
  if (hipMemcpyAsync(&h, base + fin, sizeof(MsState), hipMemcpyDeviceToHost, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return TKEF_EHIP;
  if (out) {
    out[0] = h.abar;
    out[1] = h.u;
  }
  if (cnt) {
    cnt[0] = h.k1;
    cnt[1] = h.k2;
    cnt[2] = h.rand;
    cnt[3] = h.take;
    cnt[4] = h.K1;
    cnt[5] = h.K2;
  }
  return TKEF_OK;
}


extern "C" int tkef_sparsify_execute(tkef_sparsify_plan plan, void* ws, size_t ws_bytes,
                                     int32_t* idx_out, void* val_out, uint32_t* status,
                                     hipStream_t s) {
  if (!plan) return TKEF_EINVAL;
  if (!ws || ws_bytes < plan->ws_bytes || !aligned_ws(ws)) return TKEF_EWORKSPACE;
  if (plan->bound_ws != ws) return TKEF_ESTATE;
  if (plan->k_total > 0 && (!idx_out || !val_out)) return TKEF_EINVAL;
  char* base = static_cast<char*>(ws);
  const TileDesc* tiles = reinterpret_cast<const TileDesc*>(base + plan->off_tiles);
  const GroupDesc* groups = reinterpret_cast<const GroupDesc*>(base + plan->off_groups);
  GroupState* st = reinterpret_cast<GroupState*>(base + plan->off_state);
  char* zb = base + plan->off_zero;  // the zeroed scratch
  uint32_t* hist1 = reinterpret_cast<uint32_t*>(zb + plan->off_hist1);
  uint32_t* hist2 = reinterpret_cast<uint32_t*>(zb + plan->off_hist2);
  uint16_t* summ = reinterpret_cast<uint16_t*>(base + plan->off_summ);
  const int32_t nt = plan->ntiles, ng = plan->ngroups;
  const int64_t nl = plan->nlines;
  const int lpt = plan->sel_lpt, sg = plan->sel_grid;
  const Tracer tr{plan->events, plan->n_events};
  const int val16 = plan->val_format == TKEF_VAL_F16 ? 1 : 0;
  int li = 0;  // launch index, for the timing hook
  // the last kernel clears [0, tail) of the zeroed scratch, the stream
  // [tail, zero_bytes)
  size_t tail = plan->zero_tail;
  if (plan->mode == TKEF_APPROX) {
    const int32_t last = plan->ms_passes() - 1;  // the emit kernel reads pass last's counts
    tail += (last == 0 ? 0 : ((size_t)kMsSlots * 64 + (size_t)(last - 1) * kMsRefineBins)) * 4;
  }
  uint32_t* clear_next = reinterpret_cast<uint32_t*>(zb);
  const int64_t clear_words = (int64_t)(tail / 4);
  uint32_t* stream_clear = reinterpret_cast<uint32_t*>(zb + tail);
  const int64_t stream_words = (int64_t)((plan->zero_bytes - tail) / 4);

  hipError_t e = hipSuccess;
  if (plan->needs_clear) {  // after a failed run
    e = launch_fill_u32(reinterpret_cast<uint32_t*>(zb), 0u, (int64_t)(plan->zero_bytes / 4), s);
    if (e != hipSuccess) return TKEF_EHIP;
    plan->needs_clear = false;
  }
  if (plan->mode == TKEF_APPROX) {
    MsState* ms = reinterpret_cast<MsState*>(base + plan->off_ms_state);
    uint64_t* esum = reinterpret_cast<uint64_t*>(zb + plan->off_ms_esum);
    uint32_t* emax = reinterpret_cast<uint32_t*>(zb + plan->off_ms_emax);
    uint32_t* cnt = reinterpret_cast<uint32_t*>(zb + plan->off_ms_cnt);
    uint64_t* flags = reinterpret_cast<uint64_t*>(zb + plan->off_ms_flags);
    const uint32_t k = static_cast<uint32_t>(plan->k_total);
    const int32_t N = plan->ms_rounds, passes = plan->ms_passes();
    auto rounds_of = [&](int32_t b) {
      return b == 0 ? std::min(kMsRoundsPerPass, N)
                    : std::min(kMsRoundsPerRefine,
                               N - kMsRoundsPerPass - (b - 1) * kMsRoundsPerRefine);
    };
    auto cnt_of = [&](int32_t b) {
      return b == 0 ? cnt : cnt + (size_t)kMsSlots * 64 + (size_t)(b - 1) * kMsRefineBins;
    };
    auto slots_of = [&](int32_t b) { return b == 0 ? kMsSlots : 1; };
    auto bins_of = [&](int32_t b) { return b == 0 ? 64 : kMsRefineBins; };
    e = launch_ms_stream(tiles, nt, plan->stream_grid, kMsSlots, esum, emax, summ, stream_clear,
                         stream_words, s, tr.at(li++));
    if (e == hipSuccess)
      e = launch_ms_count(tiles, nt, plan->count_grid, kMsSlots, esum, emax, summ, cnt_of(0),
                          ms, plan->d, status, s, tr.at(li++));
    for (int32_t b = 1; b < passes && e == hipSuccess; ++b)
      e = launch_ms_refine(tiles, summ, nl, lpt, sg, slots_of(b - 1), bins_of(b - 1),
                           cnt_of(b - 1), cnt_of(b), ms + b - 1, ms + b, k, plan->d,
                           rounds_of(b - 1), N, plan->ms_word, s, tr.at(li++));
    if (e == hipSuccess)
      e = launch_ms_emit(tiles, summ, nl, lpt, sg, slots_of(passes - 1), bins_of(passes - 1),
                         cnt_of(passes - 1), ms + passes - 1, ms + passes, k, plan->d,
                         rounds_of(passes - 1), N,
                         plan->ms_word, flags, idx_out, val_out, val16, status, clear_next,
                         clear_words, s, tr.at(li++));
    if (e != hipSuccess) {
      plan->needs_clear = true;
      return TKEF_EHIP;
    }
    return TKEF_OK;
  }
  if (ng == 1) {
    e = run_one_group(plan, base, zb, stream_clear, stream_words, clear_next, clear_words,
                      idx_out, val_out, val16, status, s, tr);
  } else {
    e = launch_stream(tiles, nt, plan->stream_grid, hist1, plan->nslots, summ, status,
                      stream_clear, stream_words, s, tr.at(li++));
    uint32_t* hist3 = reinterpret_cast<uint32_t*>(zb + plan->off_hist3);
    uint64_t* flags1 = reinterpret_cast<uint64_t*>(zb + plan->off_flags1);
    uint64_t* flags2 = reinterpret_cast<uint64_t*>(zb + plan->off_flags2);
    uint32_t* meta = reinterpret_cast<uint32_t*>(zb + plan->off_meta);
    uint32_t* gbase = reinterpret_cast<uint32_t*>(base + plan->off_base);
    uint32_t* cand = reinterpret_cast<uint32_t*>(base + plan->off_cand);
    if (e == hipSuccess)
      e = launch_pick(1, groups, st, hist1, plan->nslots, ng, s, tr.at(li++));
    if (e == hipSuccess)
      e = launch_gather(tiles, st, summ, nl, lpt, plan->line_grid, hist2, flags1, cand,
                        plan->cand_cap, meta, status, s, tr.at(li++));
    if (e == hipSuccess) e = launch_pick(2, groups, st, hist2, 1, ng, s, tr.at(li++));
    if (e == hipSuccess)
      e = launch_hist3(tiles, nt, st, summ, nl, lpt, plan->cand_grid, cand, meta, hist3, s,
                       tr.at(li++));
    if (e == hipSuccess) e = launch_pick(3, groups, st, hist3, 1, ng, s, tr.at(li++));
    const bool fold = ng <= emit_lds_groups();
    if (e == hipSuccess && !fold) e = launch_groupscan(groups, st, ng, gbase, s, tr.at(li++));
    if (e == hipSuccess)
      e = launch_emit(tiles, nt, groups, st, summ, nl, lpt, plan->cand_grid, cand, meta, gbase,
                      flags2, idx_out, val_out, val16, status, clear_next, clear_words,
                      fold ? ng : 0, s, tr.at(li++));
  }
  if (e != hipSuccess) {
    plan->needs_clear = true;
    return TKEF_EHIP;
  }
  return hip_rc(e);
}

extern "C" int tkef_sparsify_workspace(const int64_t* numels, int32_t ntensors, int32_t mode,
                                       double rho, int64_t k, size_t* workspace_bytes,
                                       int64_t* k_total) {
  tkef_sparsify_plan p = nullptr;
  int rc = tkef_sparsify_plan_create(numels, ntensors, mode, rho, k, &p);
  if (rc) return rc;
  rc = tkef_sparsify_plan_info(p, workspace_bytes, k_total, nullptr, nullptr, nullptr);
  tkef_sparsify_plan_destroy(p);
  return rc;
}

extern "C" int tkef_sparsify(const float* const* grads, float* const* residuals,
                             const int64_t* numels, int32_t ntensors, int32_t mode, double rho,
                             int64_t k, int32_t val_format, int32_t* idx_out, void* val_out,
                             int64_t* counts_out, void* ws, size_t ws_bytes, uint32_t* status,
                             hipStream_t stream) {
  tkef_sparsify_plan p = nullptr;
  int rc = tkef_sparsify_plan_create(numels, ntensors, mode, rho, k, &p);
  if (rc) return rc;
  rc = tkef_sparsify_plan_set_value_format(p, val_format);
  if (!rc && counts_out) rc = tkef_sparsify_plan_group_k(p, counts_out, p->ngroups);
  if (!rc) rc = tkef_sparsify_plan_bind(p, grads, residuals, ws, ws_bytes, stream);
  if (!rc) rc = tkef_sparsify_execute(p, ws, ws_bytes, idx_out, val_out, status, stream);
  tkef_sparsify_plan_destroy(p);
  return rc;
}

extern "C" int tkef_sparsify1(const float* g, float* r, int64_t d, int64_t k, int32_t* idx_out,
                              float* val_out, void* ws, size_t ws_bytes, uint32_t* status,
                              hipStream_t stream) {
  if (d < 1 || d > kMaxD || k < 1 || k > d) return TKEF_ERANGE;
  const float* gs[1] = {g};
  float* rs[1] = {r};
  return tkef_sparsify(gs, rs, &d, 1, TKEF_GLOBAL, 0.0, k, TKEF_VAL_F32, idx_out, val_out,
                       nullptr, ws, ws_bytes, status, stream);
}

extern "C" int tkef_sparsify1_static(const float* g, float* r, int64_t d, int64_t k,
                                     int32_t* idx_out, float* val_out, uint32_t* status,
                                     hipStream_t stream) {
  static_assert(TKEF_STATIC_MAX_D == kStaticMaxD && TKEF_STATIC_MAX_K == kStaticMaxK &&
                    TKEF_STATIC_SCRATCH_BYTES == kStaticScratchBytes,
                "header and library agree on the fixed scratch");
  if (!g || !r || !idx_out || !val_out) return TKEF_EINVAL;
  if (d < 1 || d > kStaticMaxD || k < 1 || k > d || k > kStaticMaxK) return TKEF_ERANGE;
  if (ranges_overlap(g, r, d)) return TKEF_EINVAL;
  // the layout of a one-tensor global plan, computed without allocating
  // (the plan's vectors stay empty)
  tkef_sparsify_plan_s p;
  p.ntensors = 1;
  p.mode = TKEF_GLOBAL;
  p.ngroups = 1;
  p.d = d;
  p.k_total = k;
  p.ntiles = (int32_t)((d + kTile - 1) / kTile);
  p.nlines = (int64_t)p.ntiles * kLinesPerTile;
  if (!sparsify_layout(&p)) return TKEF_ERANGE;
  if (p.ws_bytes > kStaticScratchBytes) return TKEF_EWORKSPACE;  // (not within the limits)
  if (stream_grid_for(p.ntiles, &p.stream_grid, nullptr)) return TKEF_EHIP;
  hipError_t e = hipSuccess;
  char* base = static_cast<char*>(static_scratch(&e));
  if (!base) return TKEF_EHIP;
  // the array keeps the previous call's contents: the set-up kernel writes
  // the tables, clears the histograms and the last tile's line summaries
  // (the stream rewrites the summaries of every line that holds elements)
  char* zb = base + p.off_zero;
  uint16_t* summ = reinterpret_cast<uint16_t*>(base + p.off_summ);
  e = launch_setup_one(reinterpret_cast<TileDesc*>(base + p.off_tiles),
                       reinterpret_cast<GroupDesc*>(base + p.off_groups), g, r, d, k, p.ntiles,
                       reinterpret_cast<uint32_t*>(zb), (int64_t)(p.zero_bytes / 4),
                       reinterpret_cast<uint32_t*>(summ + (int64_t)(p.ntiles - 1) * kLinesPerTile),
                       kLinesPerTile / 2, stream);
  if (e == hipSuccess)
    e = run_one_group(&p, base, zb, nullptr, 0, nullptr, 0, idx_out, val_out, 0, status,
                      stream, Tracer{nullptr, 0});
  return hip_rc(e);
}

// ============================================================================
// update plan

static const char* const kUpdateLaunches[] = {"seg", "update"};
constexpr int32_t kUpdateNLaunch = 2;
// LARS executions: the fused sparse update (seg, norms, rates, step) and the
// rates from dense gradients (norms, rates)
static const char* const kLarsLaunches[] = {"seg", "lars_norm", "lars_rates", "lars_step"};
static const char* const kLarsDenseLaunches[] = {"lars_norm_dense", "lars_rates"};

struct tkef_update_plan_s {
  int32_t ntensors = 0, P = 0, ntiles_u = 0;
  int64_t d = 0, stride = 0;
  std::vector<int64_t> numels, goff;
  std::vector<UpdTensor> tens;
  std::vector<int32_t> tile_first;
  std::vector<int32_t> tpair;  // LARS: first (tile, tensor) pair of each tensor; [T] = pairs
  size_t off_tens = 0, off_first = 0, off_seg = 0, off_tpair = 0, off_part = 0, off_rate = 0,
         off_gptr = 0, off_lists = 0, ws_bytes = 0;
  bool table = false;  // lists given as per-worker pointers (WorkerList table in ws)
  void* bound_ws = nullptr;
  bool has_mom = false;
  bool has_grads = false;  // dense gradients bound (LARS rates)
  int32_t val_format = TKEF_VAL_F32;  // value arrays read by execute / aggregate
  bool det = false;  // sums in worker order (tkef_update_plan_set_deterministic)
  hipEvent_t* events = nullptr;
  int32_t n_events = 0;
};

namespace {

int update_plan_create(const int64_t* numels, int32_t ntensors, int32_t P, int64_t stride,
                       bool table, tkef_update_plan* plan_out) {
  if (!plan_out) return TKEF_EINVAL;
  *plan_out = nullptr;
  int64_t d = 0;
  int rc = check_numels(numels, ntensors, &d);
  if (rc) return rc;
  if (P < 1 || P > 65535) return TKEF_EINVAL;
  if (stride < 0 || stride > kMaxD) return TKEF_ERANGE;
  if ((int64_t)P * stride > (int64_t)1 << 40) return TKEF_ERANGE;
  tkef_update_plan p = new (std::nothrow) tkef_update_plan_s();
  if (!p) return TKEF_ENOMEM;
  try {
    p->ntensors = ntensors;
    p->P = P;
    p->d = d;
    p->stride = stride;
    p->numels.assign(numels, numels + ntensors);
    p->goff.resize(ntensors);
    int64_t off = 0;
    for (int32_t t = 0; t < ntensors; ++t) {
      p->goff[t] = off;
      off += numels[t];
    }
    p->ntiles_u = static_cast<int32_t>((d + kUTile - 1) / kUTile);
    // tile_first[u]: the tensor holding position u * kUTile; [ntiles_u] = T
    p->tile_first.assign(p->ntiles_u + 1, ntensors);
    int32_t t = 0;
    for (int32_t u = 0; u < p->ntiles_u; ++u) {
      const int64_t pos = (int64_t)u * kUTile;
      while (t < ntensors && p->goff[t] + numels[t] <= pos) ++t;
      p->tile_first[u] = t;
    }
    // LARS pairs: tensor t overlaps update tiles goff_t >> kUShift ..
    // (goff_t + n_t - 1) >> kUShift
    p->tpair.assign(ntensors + 1, 0);
    for (int32_t t = 0; t < ntensors; ++t) {
      const int64_t n = numels[t];
      const int64_t tiles = n > 0 ? ((p->goff[t] + n - 1) >> kUShift) - (p->goff[t] >> kUShift) + 1
                                  : 0;
      p->tpair[t + 1] = p->tpair[t] + (int32_t)tiles;
    }
    p->tens.resize(ntensors);
    size_t o = 0;
    p->off_tens = o;   o = align_up(o + p->tens.size() * sizeof(UpdTensor));
    p->off_first = o;  o = align_up(o + p->tile_first.size() * sizeof(int32_t));
    p->off_seg = o;    o = align_up(o + (size_t)P * (p->ntiles_u + 1) * sizeof(int32_t));
    p->off_tpair = o;  o = align_up(o + p->tpair.size() * sizeof(int32_t));
    p->off_part = o;   o = align_up(o + (size_t)p->tpair[ntensors] * 16);
    p->off_rate = o;   o = align_up(o + (size_t)ntensors * sizeof(double));
    p->off_gptr = o;   o = align_up(o + (size_t)ntensors * sizeof(float*));
    p->table = table;
    if (table) {
      p->off_lists = o;  o = align_up(o + (size_t)P * sizeof(WorkerList));
    }
    p->ws_bytes = o;
  } catch (const std::bad_alloc&) {
    delete p;
    return TKEF_ENOMEM;
  }
  *plan_out = p;
  return TKEF_OK;
}

}  // namespace

extern "C" int tkef_update_plan_create(const int64_t* numels, int32_t ntensors, int32_t P,
                                       int64_t stride, tkef_update_plan* plan_out) {
  return update_plan_create(numels, ntensors, P, stride, false, plan_out);
}

extern "C" int tkef_update_plan_destroy(tkef_update_plan plan) {
  delete plan;
  return TKEF_OK;
}

extern "C" int tkef_update_plan_info(tkef_update_plan plan, size_t* workspace_bytes,
                                     int64_t* d_total, int32_t* nlaunch) {
  if (!plan) return TKEF_EINVAL;
  if (workspace_bytes) *workspace_bytes = plan->ws_bytes;
  if (d_total) *d_total = plan->d;
  if (nlaunch) *nlaunch = kUpdateNLaunch;
  return TKEF_OK;
}

namespace {

// The checks of tkef_update_plan_bind (nothing is enqueued before them).
int check_update_bind(tkef_update_plan plan, float* const* params, float* const* momentum,
                      void* ws, size_t ws_bytes) {
  if (!plan || !params) return TKEF_EINVAL;
  if (!ws || !aligned_ws(ws) || ws_bytes < plan->ws_bytes) return TKEF_EWORKSPACE;
  for (int32_t t = 0; t < plan->ntensors; ++t) {
    const int64_t n = plan->numels[t];
    if (n == 0) continue;
    if (!params[t]) return TKEF_EINVAL;
    if (momentum) {
      if (!momentum[t]) return TKEF_EINVAL;
      if (ranges_overlap(params[t], momentum[t], n)) return TKEF_EINVAL;
    }
  }
  return TKEF_OK;
}

}  // namespace

extern "C" int tkef_update_plan_bind(tkef_update_plan plan, float* const* params,
                                     float* const* momentum, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
  const int rc = check_update_bind(plan, params, momentum, ws, ws_bytes);
  if (rc) return rc;
  for (int32_t t = 0; t < plan->ntensors; ++t) {
    plan->tens[t].w = params[t];
    plan->tens[t].b = momentum ? momentum[t] : nullptr;
    plan->tens[t].goff = plan->goff[t];
    plan->tens[t].n = plan->numels[t];
  }
  char* base = static_cast<char*>(ws);
  hipError_t e = hipMemcpyAsync(base + plan->off_tens, plan->tens.data(),
                                plan->tens.size() * sizeof(UpdTensor), hipMemcpyHostToDevice,
                                stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(base + plan->off_first, plan->tile_first.data(),
                       plan->tile_first.size() * sizeof(int32_t), hipMemcpyHostToDevice,
                       stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(base + plan->off_tpair, plan->tpair.data(),
                       plan->tpair.size() * sizeof(int32_t), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    plan->bound_ws = nullptr;
    return TKEF_EHIP;
  }
  plan->bound_ws = ws;
  plan->has_mom = momentum != nullptr;
  plan->has_grads = false;
  return TKEF_OK;
}

extern "C" int tkef_update_plan_bind_grads(tkef_update_plan plan, const float* const* grads,
                                           void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!plan || !grads) return TKEF_EINVAL;
  if (!ws || ws_bytes < plan->ws_bytes || !aligned_ws(ws)) return TKEF_EWORKSPACE;
  if (plan->bound_ws != ws) return TKEF_ESTATE;
  std::vector<const float*> g(plan->ntensors, nullptr);
  for (int32_t t = 0; t < plan->ntensors; ++t) {
    if (plan->numels[t] == 0) continue;
    if (!grads[t]) return TKEF_EINVAL;
    g[t] = grads[t];
  }
  char* base = static_cast<char*>(ws);
  hipError_t e = hipMemcpyAsync(base + plan->off_gptr, g.data(), g.size() * sizeof(float*),
                                hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return TKEF_EHIP;
  plan->has_grads = true;
  return TKEF_OK;
}

extern "C" int tkef_update_plan_set_events(tkef_update_plan plan, hipEvent_t* events,
                                           int32_t n_events) {
  if (!plan || n_events < 0 || (events && n_events == 0)) return TKEF_EINVAL;
  plan->events = events;
  plan->n_events = events ? n_events : 0;
  return TKEF_OK;
}

extern "C" const char* tkef_update_plan_launch_name(tkef_update_plan plan, int32_t i) {
  if (!plan || i < 0 || i >= kUpdateNLaunch) return nullptr;
  return kUpdateLaunches[i];
}

extern "C" int tkef_update_plan_set_value_format(tkef_update_plan plan, int32_t format) {
  if (!plan || (format != TKEF_VAL_F32 && format != TKEF_VAL_F16)) return TKEF_EINVAL;
  plan->val_format = format;
  return TKEF_OK;
}

extern "C" int tkef_update_plan_set_deterministic(tkef_update_plan plan, int32_t on) {
  if (!plan || (on != 0 && on != 1)) return TKEF_EINVAL;
  if (plan->table) return TKEF_EINVAL;  // (the per-worker pointer form sums in any order)
  plan->det = on != 0;
  return TKEF_OK;
}

namespace {

// seg + update with the given operation on the tile sums.
int update_run(tkef_update_plan plan, const int32_t* idx, const void* val, const int32_t* nnz,
               float lr, float mu, float wd, int op, void* ws, size_t ws_bytes,
               uint32_t* status, hipStream_t s) {
  if (!plan) return TKEF_EINVAL;
  if (!ws || ws_bytes < plan->ws_bytes || !aligned_ws(ws)) return TKEF_EWORKSPACE;
  if (plan->bound_ws != ws) return TKEF_ESTATE;
  if (plan->stride > 0 && (!idx || !val)) return TKEF_EINVAL;
  char* base = static_cast<char*>(ws);
  const UpdTensor* tens = reinterpret_cast<const UpdTensor*>(base + plan->off_tens);
  const int32_t* first = reinterpret_cast<const int32_t*>(base + plan->off_first);
  int32_t* seg = reinterpret_cast<int32_t*>(base + plan->off_seg);
  const int has_mom = (op == kOpSgd && mu != 0.0f) ? 1 : 0;
  const int val16 = plan->val_format == TKEF_VAL_F16 ? 1 : 0;
  const Tracer tr{plan->events, plan->n_events};
  hipError_t e = launch_seg(idx, plan->stride, nnz, plan->P, (int32_t)plan->d, plan->ntiles_u,
                            seg, status, s, tr.at(0));
  if (e == hipSuccess)
    e = launch_update(tens, first, plan->ntensors, (int32_t)plan->d, plan->ntiles_u, idx, val,
                      val16, plan->stride, nnz, plan->P, seg, lr, mu, wd, op, has_mom,
                      LarsArgs{nullptr, nullptr, nullptr, 0.0f}, plan->det, s, tr.at(1));
  return hip_rc(e);
}

bool finite_all(double a, double b, double c) {
  return std::isfinite(a) && std::isfinite(b) && std::isfinite(c);
}

}  // namespace

extern "C" int tkef_update_execute(tkef_update_plan plan, const int32_t* idx, const void* val,
                                   const int32_t* nnz, float lr, float mu, float wd, void* ws,
                                   size_t ws_bytes, uint32_t* status, hipStream_t s) {
  if (!plan) return TKEF_EINVAL;
  if (!std::isfinite(lr) || !std::isfinite(mu) || !std::isfinite(wd)) return TKEF_ERANGE;
  if (mu != 0.0f && !plan->has_mom) return TKEF_EINVAL;
  const int op = (mu == 0.0f && wd == 0.0f) ? kOpSparseSgd : kOpSgd;
  return update_run(plan, idx, val, nnz, lr, mu, wd, op, ws, ws_bytes, status, s);
}

extern "C" int tkef_aggregate_execute(tkef_update_plan plan, const int32_t* idx, const void* val,
                                      const int32_t* nnz, void* ws, size_t ws_bytes,
                                      uint32_t* status, hipStream_t s) {
  return update_run(plan, idx, val, nnz, 0.0f, 0.0f, 0.0f, kOpAggregate, ws, ws_bytes, status, s);
}

extern "C" int tkef_lars_update_execute(tkef_update_plan plan, const int32_t* idx,
                                        const void* val, const int32_t* nnz, double gamma,
                                        double eta, double eps, float mu, double* rate_out,
                                        void* ws, size_t ws_bytes, uint32_t* status,
                                        hipStream_t s) {
  if (!plan) return TKEF_EINVAL;
  if (!finite_all(gamma, eta, eps) || !(eps >= 0.0) || !std::isfinite(mu)) return TKEF_ERANGE;
  if (mu != 0.0f && !plan->has_mom) return TKEF_EINVAL;
  if (!ws || ws_bytes < plan->ws_bytes || !aligned_ws(ws)) return TKEF_EWORKSPACE;
  if (plan->bound_ws != ws) return TKEF_ESTATE;
  if (plan->stride > 0 && (!idx || !val)) return TKEF_EINVAL;
  char* base = static_cast<char*>(ws);
  const UpdTensor* tens = reinterpret_cast<const UpdTensor*>(base + plan->off_tens);
  const int32_t* first = reinterpret_cast<const int32_t*>(base + plan->off_first);
  int32_t* seg = reinterpret_cast<int32_t*>(base + plan->off_seg);
  const int32_t* tpair = reinterpret_cast<const int32_t*>(base + plan->off_tpair);
  double2* part = reinterpret_cast<double2*>(base + plan->off_part);
  double* rate = reinterpret_cast<double*>(base + plan->off_rate);
  const int has_mom = mu != 0.0f ? 1 : 0;
  const int val16 = plan->val_format == TKEF_VAL_F16 ? 1 : 0;
  const float eps32 = static_cast<float>(eps);
  const Tracer tr{plan->events, plan->n_events};
  const int32_t d = (int32_t)plan->d, T = plan->ntensors;
  hipError_t e = launch_seg(idx, plan->stride, nnz, plan->P, d, plan->ntiles_u, seg, status, s,
                            tr.at(0));
  if (e == hipSuccess)
    e = launch_update(tens, first, T, d, plan->ntiles_u, idx, val, val16, plan->stride, nnz,
                      plan->P, seg, 0.0f, 0.0f, 0.0f, kOpLarsNorm, 0,
                      LarsArgs{part, tpair, nullptr, eps32}, plan->det, s, tr.at(1));
  if (e == hipSuccess)
    e = launch_lars_rates(tpair, part, T, gamma, eta, eps, rate, rate_out, s, tr.at(2));
  if (e == hipSuccess)
    e = launch_update(tens, first, T, d, plan->ntiles_u, idx, val, val16, plan->stride, nnz,
                      plan->P, seg, 0.0f, mu, 0.0f, kOpLarsApply, has_mom,
                      LarsArgs{part, tpair, rate, eps32}, plan->det, s, tr.at(3));
  return hip_rc(e);
}

extern "C" int tkef_lars_rates_execute(tkef_update_plan plan, double gamma, double eta,
                                       double eps, double* rate_out, void* ws, size_t ws_bytes,
                                       hipStream_t s) {
  if (!plan) return TKEF_EINVAL;
  if (!finite_all(gamma, eta, eps) || !(eps >= 0.0)) return TKEF_ERANGE;
  if (!ws || ws_bytes < plan->ws_bytes || !aligned_ws(ws)) return TKEF_EWORKSPACE;
  if (plan->bound_ws != ws || !plan->has_grads) return TKEF_ESTATE;
  char* base = static_cast<char*>(ws);
  const UpdTensor* tens = reinterpret_cast<const UpdTensor*>(base + plan->off_tens);
  const int32_t* first = reinterpret_cast<const int32_t*>(base + plan->off_first);
  const int32_t* tpair = reinterpret_cast<const int32_t*>(base + plan->off_tpair);
  double2* part = reinterpret_cast<double2*>(base + plan->off_part);
  double* rate = reinterpret_cast<double*>(base + plan->off_rate);
  const float* const* gptrs = reinterpret_cast<const float* const*>(base + plan->off_gptr);
  const Tracer tr{plan->events, plan->n_events};
  hipError_t e = launch_lars_norm_dense(tens, gptrs, first, plan->ntensors, (int32_t)plan->d,
                                        plan->ntiles_u, part, tpair, s, tr.at(0));
  if (e == hipSuccess)
    e = launch_lars_rates(tpair, part, plan->ntensors, gamma, eta, eps, rate, rate_out, s,
                          tr.at(1));
  return hip_rc(e);
}

extern "C" const char* tkef_lars_launch_name(int32_t dense, int32_t i) {
  if (dense == 1) return (i >= 0 && i < 2) ? kLarsDenseLaunches[i] : nullptr;
  if (dense == 0) return (i >= 0 && i < 4) ? kLarsLaunches[i] : nullptr;
  return nullptr;
}

extern "C" int tkef_update_workspace(const int64_t* numels, int32_t ntensors, int32_t P,
                                     int64_t stride, size_t* workspace_bytes) {
  tkef_update_plan p = nullptr;
  int rc = tkef_update_plan_create(numels, ntensors, P, stride, &p);
  if (rc) return rc;
  rc = tkef_update_plan_info(p, workspace_bytes, nullptr, nullptr);
  tkef_update_plan_destroy(p);
  return rc;
}

extern "C" int tkef_sparse_aggregate_update(float* const* params, float* const* momentum,
                                            const int64_t* numels, int32_t ntensors,
                                            const int32_t* idx, const void* val, int32_t P,
                                            int64_t stride, const int32_t* nnz, float lr,
                                            float mu, float wd, void* ws, size_t ws_bytes,
                                            uint32_t* status, hipStream_t stream) {
  tkef_update_plan p = nullptr;
  int rc = tkef_update_plan_create(numels, ntensors, P, stride, &p);
  if (rc) return rc;
  rc = tkef_update_plan_bind(p, params, momentum, ws, ws_bytes, stream);
  if (!rc) rc = tkef_update_execute(p, idx, val, nnz, lr, mu, wd, ws, ws_bytes, status, stream);
  tkef_update_plan_destroy(p);
  return rc;
}

extern "C" int tkef_sparse_aggregate(float* const* outs, const int64_t* numels, int32_t ntensors,
                                     const int32_t* idx, const void* val, int32_t val_format,
                                     int32_t P, int64_t stride, const int32_t* nnz, void* ws,
                                     size_t ws_bytes, uint32_t* status, hipStream_t stream) {
  tkef_update_plan p = nullptr;
  int rc = tkef_update_plan_create(numels, ntensors, P, stride, &p);
  if (rc) return rc;
  rc = tkef_update_plan_set_value_format(p, val_format);
  if (!rc) rc = tkef_update_plan_bind(p, outs, nullptr, ws, ws_bytes, stream);
  if (!rc) rc = tkef_aggregate_execute(p, idx, val, nnz, ws, ws_bytes, status, stream);
  tkef_update_plan_destroy(p);
  return rc;
}

extern "C" int tkef_aggregate_workspace(const int64_t* numels, int32_t ntensors, int32_t P,
                                        size_t* workspace_bytes) {
  tkef_update_plan p = nullptr;
  int rc = update_plan_create(numels, ntensors, P, 0, true, &p);
  if (rc) return rc;
  rc = tkef_update_plan_info(p, workspace_bytes, nullptr, nullptr);
  tkef_update_plan_destroy(p);
  return rc;
}

extern "C" int tkef_aggregate_update(float* const* params, float* const* momentum,
                                     const int64_t* numels, int32_t ntensors,
                                     const int32_t* const* idx, const float* const* val,
                                     const int64_t* nnz, int32_t P, float lr, float mu, float wd,
                                     void* ws, size_t ws_bytes, uint32_t* status,
                                     hipStream_t stream) {
  if (!idx || !val || !nnz || P < 1) return TKEF_EINVAL;
  if (!std::isfinite(lr) || !std::isfinite(mu) || !std::isfinite(wd)) return TKEF_ERANGE;
  if (mu != 0.0f && !momentum) return TKEF_EINVAL;
  std::vector<WorkerList> lists;
  int64_t max_n = 0;
  try {
    lists.resize(P);
  } catch (const std::bad_alloc&) {
    return TKEF_ENOMEM;
  }
  for (int32_t q = 0; q < P; ++q) {
    if (nnz[q] < 0) return TKEF_EINVAL;
    if (nnz[q] > kMaxD) return TKEF_ERANGE;
    if (nnz[q] > 0 && (!idx[q] || !val[q])) return TKEF_EINVAL;
    lists[q] = WorkerList{idx[q], val[q], nnz[q], 0};
    max_n = std::max(max_n, nnz[q]);
  }
  tkef_update_plan p = nullptr;
  int rc = update_plan_create(numels, ntensors, P, 0, true, &p);
  if (rc) return rc;
  rc = check_update_bind(p, params, momentum, ws, ws_bytes);
  if (rc) {
    tkef_update_plan_destroy(p);
    return rc;
  }
  // the worker table goes in first; bind's synchronization covers its copy
  char* base = static_cast<char*>(ws);
  if (hipMemcpyAsync(base + p->off_lists, lists.data(), lists.size() * sizeof(WorkerList),
                     hipMemcpyHostToDevice, stream) != hipSuccess) {
    tkef_update_plan_destroy(p);
    return TKEF_EHIP;
  }
  rc = tkef_update_plan_bind(p, params, momentum, ws, ws_bytes, stream);
  if (!rc) {
    const UpdTensor* tens = reinterpret_cast<const UpdTensor*>(base + p->off_tens);
    const int32_t* first = reinterpret_cast<const int32_t*>(base + p->off_first);
    int32_t* seg = reinterpret_cast<int32_t*>(base + p->off_seg);
    const WorkerList* table = reinterpret_cast<const WorkerList*>(base + p->off_lists);
    const int op = (mu == 0.0f && wd == 0.0f) ? kOpSparseSgd : kOpSgd;
    const int has_mom = mu != 0.0f ? 1 : 0;
    hipError_t e = launch_seg_table(table, P, max_n, (int32_t)p->d, p->ntiles_u, seg, status,
                                    stream, Ev{});
    if (e == hipSuccess)
      e = launch_update_table(tens, first, p->ntensors, (int32_t)p->d, p->ntiles_u, table, P,
                              seg, lr, mu, wd, op, has_mom, stream, Ev{});
    rc = hip_rc(e);
  }
  tkef_update_plan_destroy(p);
  return rc;
}

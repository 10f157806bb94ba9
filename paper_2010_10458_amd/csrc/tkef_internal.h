// Internal layout shared by the host library and the gfx950 kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace tkef {

// ---- sparsify tiling --------------------------------------------------------
// A tile is up to kTile consecutive elements of one tensor. A line is kLine
// consecutive elements (one 128-B cache line of float32) and gets a 16-bit
// summary: the top 15 bits of the largest magnitude key in it. Tile i owns
// summary entries [i * kLinesPerTile, (i + 1) * kLinesPerTile).
constexpr int kBlock = 256;
constexpr int kTile = 8192;
constexpr int kLine = 32;
constexpr int kLinesPerTile = kTile / kLine;  // == kBlock: one line per thread
// A sparsify tensor list may take at most kMaxTiles tiles (tensor t takes
// ceil(numel_t / kTile)): the selection grids cover at most that many tiles'
// summary lines, and the per-tensor and MSTopK selections carry a candidate as
// (tile << 13) | position-in-tile in 32 bits. One tensor of 2^31 - 1
// elements takes exactly kMaxTiles.
constexpr int64_t kMaxTiles = (int64_t)1 << 18;
static_assert(kMaxTiles * kTile <= (int64_t)1 << 32, "candidate code width");
static_assert(kLinesPerTile == kBlock, "one summary line per thread");
// The stream walks the tiles in units of kStreamUnit elements (a persistent
// grid takes units round-robin).
constexpr int kStreamUnit = 2048;

// Magnitude key = float bits with the sign cleared. The threshold search is a
// three-level radix select on it: 11 bits, then 10, then 10.
constexpr int kH1Bins = 2048, kH1Shift = 20;
constexpr int kH2Bins = 1024, kH2Shift = 10;
constexpr int kH3Bins = 1024;
// copies of the level-1 histogram (the stream's workgroups add into copy
// blockIdx % copies): one global selection, per-tensor selections
constexpr int kSlotsOne = 4, kSlotsMany = 4;

struct TileDesc {        // 32 B, one per tile, written at bind
  const float* g;        // gradient, first element of the tile
  float* r;              // residual, first element of the tile
  int32_t gstart;        // global position of the first element
  int32_t len;           // elements in the tile, 1..kTile
  int32_t group;         // selection group
  int32_t reserved;
};
static_assert(sizeof(TileDesc) == 32, "TileDesc layout");

struct GroupDesc {       // one per selection group, written at bind
  uint32_t k;            // pairs the group selects
  uint32_t tile_begin;   // first tile of the group
  uint32_t out_base;     // first output slot of the group
  uint32_t pad;
};

struct GroupState {      // per group, rewritten by every execution
  uint32_t need;         // still to take from the current key class
  uint32_t prefix;       // key bits fixed so far
  uint32_t T;            // final threshold key
  uint32_t n_eq;         // elements with key == T
};

// ---- approximate selection (MSTopK) ------------------------------------------
// State of one MSTopK run between counting passes: the mean and maximum of
// |x|, the bisection bracket [l, r] of the ratio, the recorded counts and
// their threshold keys, and (after the last round) the window.
struct MsState {
  double abar, u, l, r;
  uint32_t k1, k2;       // largest count <= k, smallest count > k (start 0, d)
  uint32_t K1, K2;       // their threshold keys (start: none = 2^31, 0)
  uint32_t rand, take;   // window offset in the band, elements taken from it
  uint32_t level, bad;   // rounds done; non-finite input seen
};
constexpr int kMsRoundsPerPass = 6;     // first pass: 63 thresholds = six bisection rounds
constexpr int kMsRoundsPerRefine = 12;  // later passes: 4095 thresholds = twelve rounds
constexpr int kMsRefineBins = 1 << kMsRoundsPerRefine;
constexpr int kMsMaxRounds = 48;        // ratios stay exact dyadic doubles
constexpr int kMsSlots = 16;          // copies of the per-pass totals
constexpr int kMsDigitStride = 16;    // words per copy of the exact-sum digits

// ---- update tiling ------------------------------------------------------------
// Update tiles are aligned blocks of kUTile global positions; one workgroup
// accumulates a tile's sparse contributions in LDS and then applies the SGD
// step to the parameters (and momentum) of that range.
constexpr int kUBlock = 256;
constexpr int kUShift = 12;
constexpr int kUTile = 1 << kUShift;  // 4096 positions, 16 KB of LDS

// what the update kernel does with the tile sums G
enum { kOpSgd = 0, kOpSparseSgd = 1, kOpAggregate = 2, kOpLarsNorm = 3, kOpLarsApply = 4 };

// LARS (Eq. lars): per (update tile, tensor) pair the partial sums of w^2 and
// G^2 (double); pairs are tensor-major, tensor t owning [tpair[t],
// tpair[t + 1]), one per update tile it overlaps, in tile order. rate[t] is
// the tensor's rate (double).
struct LarsArgs {
  double2* part;
  const int32_t* tpair;
  const double* rate;
  float eps;
};

struct UpdTensor {       // 32 B, one per parameter tensor, written at bind
  float* w;
  float* b;              // momentum buffer or null
  int64_t goff;          // global position of element 0
  int64_t n;
};
static_assert(sizeof(UpdTensor) == 32, "UpdTensor layout");

// One worker's list in the per-worker pointer form of the aggregate: n
// entries at idx[0..n) (ascending positions) and val[0..n) (binary32).
struct WorkerList {      // 32 B, one per worker, written by the call
  const int32_t* idx;
  const void* val;
  int64_t n;
  int64_t reserved;
};
static_assert(sizeof(WorkerList) == 32, "WorkerList layout");

// ---- fixed scratch for callers that cannot allocate --------------------------
// One single-tensor exact selection of d <= kStaticMaxD elements with
// k <= kStaticMaxK needs at most 35.1 MiB of workspace (checked over every
// tile count by the host tests); the array holds 36 MiB.
constexpr int64_t kStaticMaxD = (int64_t)1 << 26;
constexpr int64_t kStaticMaxK = (int64_t)1 << 17;
constexpr size_t kStaticScratchBytes = (size_t)36 << 20;
// Device address of the current device's copy of the fixed scratch array
// (looked up once per device with hipGetSymbolAddress); null on failure, with
// the HIP error in *err.
void* static_scratch(hipError_t* err);
// Writes the tile table and group descriptor of one tensor of d elements
// (k pairs) into the workspace, and zeroes n_zero words at zero and
// n_tail words at tail.
hipError_t launch_setup_one(TileDesc* tiles, GroupDesc* groups, const float* g, float* r,
                            int64_t d, int64_t k, int32_t ntiles, uint32_t* zero, int64_t n_zero,
                            uint32_t* tail, int64_t n_tail, hipStream_t s);

// ---- kernel launchers (tkef_kernels.hip) --------------------------------------
// Optional timing events attached to one launch (recorded by the dispatch
// itself at the kernel's start and end).
struct Ev {
  hipEvent_t start = nullptr, stop = nullptr;
};
// Each returns the hipError_t of its launch.
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
// clear / clear_words: scratch the stream zeroes for the later kernels of the
// execution (it does not use it itself)
hipError_t launch_stream(const TileDesc* tiles, int32_t ntiles, int32_t grid, uint32_t* hist1,
                         int32_t nslots, uint16_t* summ, uint32_t* status, uint32_t* clear,
                         int64_t clear_words, hipStream_t s, const Ev& ev);
hipError_t launch_pick(int level, const GroupDesc* groups, GroupState* st,
                       const uint32_t* hist, int32_t nslots, int32_t ngroups, hipStream_t s, const Ev& ev);
// one selection group
constexpr int kPerBin = 4;  // band keys per (level-2 bin, region) kept in the rbin table
// block: collect_block(nlines, k, d) threads per workgroup
hipError_t launch_collect(const TileDesc* tiles, const GroupDesc* groups, GroupState* st,
                          const uint32_t* hist1, int nslots, const uint16_t* summ, int64_t nlines,
                          int lpt, int32_t grid, int32_t block, uint32_t rcap, uint32_t* hist2,
                          uint32_t* rbin, uint32_t* rcand, uint32_t* rband, uint32_t* rbtmp,
                          uint32_t* rsuf, uint32_t* rcnt, hipStream_t s, const Ev& ev);
hipError_t launch_finish(const TileDesc* tiles, const GroupDesc* groups,
                         const GroupState* st, const uint16_t* summ, int64_t nlines, int lpt,
                         int32_t grid, int32_t block, uint32_t rcap, const uint32_t* hist2,
                         const uint32_t* rbin, const uint32_t* rcand, const uint32_t* rband,
                         const uint32_t* rsuf,
                         const uint32_t* rcnt, int32_t* idx_out, void* val_out, int val16,
                         uint32_t* clear_next, int64_t clear_words, uint32_t* ticket,
                         uint32_t* rzr, hipStream_t s, const Ev& ev);
// several selection groups
hipError_t launch_gather(const TileDesc* tiles, const GroupState* st, const uint16_t* summ,
                         int64_t nlines, int lpt, int32_t grid, uint32_t* hist2, uint64_t* flags,
                         uint32_t* cand, uint32_t cap, uint32_t* meta, uint32_t* status,
                         hipStream_t s, const Ev& ev);
hipError_t launch_hist3(const TileDesc* tiles, int32_t ntiles, const GroupState* st,
                        const uint16_t* summ, int64_t nlines, int lpt, int32_t grid,
                        const uint32_t* cand, const uint32_t* meta, uint32_t* hist3,
                        hipStream_t s, const Ev& ev);
hipError_t launch_groupscan(const GroupDesc* groups, const GroupState* st, int32_t ngroups,
                            uint32_t* base, hipStream_t s, const Ev& ev);
hipError_t launch_emit(const TileDesc* tiles, int32_t ntiles, const GroupDesc* groups,
                       const GroupState* st, const uint16_t* summ, int64_t nlines, int lpt,
                       int32_t grid, const uint32_t* cand, const uint32_t* meta,
                       const uint32_t* base, uint64_t* flags, int32_t* idx_out, void* val_out,
                       int val16, uint32_t* status, uint32_t* clear_next, int64_t clear_words,
                       int32_t fold_ngroups, hipStream_t s, const Ev& ev);
// MSTopK (one group, TKEF_APPROX). st[b] = state before pass b (written by
// pass b's kernel), st[passes] = the final state (written by emit).
hipError_t launch_ms_stream(const TileDesc* tiles, int32_t ntiles, int32_t grid, int32_t nslots,
                            uint64_t* esum, uint32_t* emax, uint16_t* summ, uint32_t* clear,
                            int64_t clear_words, hipStream_t s,
                            const Ev& ev);
hipError_t launch_ms_count(const TileDesc* tiles, int32_t ntiles, int32_t grid, int32_t nslots,
                           const uint64_t* esum, const uint32_t* emax, const uint16_t* summ,
                           uint32_t* cnt, MsState* st_out, int64_t d, uint32_t* status,
                           hipStream_t s, const Ev& ev);
// The previous pass left prev_slots copies of prev_nb counters at cnt_prev
// (the first pass: kMsSlots x 64, a refine pass: 1 x kMsRefineBins).
hipError_t launch_ms_refine(const TileDesc* tiles, const uint16_t* summ, int64_t nlines, int lpt,
                            int32_t grid, int32_t prev_slots, int32_t prev_nb,
                            const uint32_t* cnt_prev, uint32_t* cnt, const MsState* st_prev,
                            MsState* st_out, uint32_t k, int64_t d, int32_t rounds_prev,
                            int32_t n_search, uint64_t window_word, hipStream_t s,
                            const Ev& ev);
hipError_t launch_ms_emit(const TileDesc* tiles, const uint16_t* summ, int64_t nlines, int lpt,
                          int32_t grid, int32_t prev_slots, int32_t prev_nb,
                          const uint32_t* cnt_prev, const MsState* st_prev, MsState* st_out,
                          uint32_t k, int64_t d, int32_t rounds_prev, int32_t n_search,
                          uint64_t window_word, uint64_t* flags, int32_t* idx_out,
                          void* val_out, int val16, uint32_t* status, uint32_t* clear_next,
                          int64_t clear_words, hipStream_t s, const Ev& ev);
// launch-shape limits of the selection kernels
int32_t select_max_groups();
int32_t select_block();
// threads per workgroup of collect and finish (one exact selection group)
int32_t collect_block(int64_t nlines, int64_t k, int64_t d);
int32_t select_max_lpt();
int32_t emit_lds_groups();  // groups whose bases k_emit can form itself

hipError_t launch_seg(const int32_t* idx, int64_t stride, const int32_t* nnz, int32_t P,
                      int32_t d, int32_t ntiles_u, int32_t* seg, uint32_t* status,
                      hipStream_t s, const Ev& ev);
hipError_t launch_update(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                         int32_t d, int32_t ntiles_u, const int32_t* idx, const void* val,
                         int val16, int64_t stride, const int32_t* nnz, int32_t P,
                         const int32_t* seg, float lr, float mu, float wd, int op, int has_mom,
                         const LarsArgs& lars, bool det, hipStream_t s, const Ev& ev);
// the same two steps over P per-worker lists (table in device memory; max_n:
// the longest list)
hipError_t launch_seg_table(const WorkerList* lists, int32_t P, int64_t max_n, int32_t d,
                            int32_t ntiles_u, int32_t* seg, uint32_t* status, hipStream_t s,
                            const Ev& ev);
hipError_t launch_update_table(const UpdTensor* tens, const int32_t* tile_first, int32_t ntens,
                               int32_t d, int32_t ntiles_u, const WorkerList* lists, int32_t P,
                               const int32_t* seg, float lr, float mu, float wd, int op,
                               int has_mom, hipStream_t s, const Ev& ev);
// LARS: partial sums of w^2 and g^2 from dense gradients (g pointer per
// tensor), and the per-tensor rates from the partial sums
hipError_t launch_lars_norm_dense(const UpdTensor* tens, const float* const* gptrs,
                                  const int32_t* tile_first, int32_t ntens, int32_t d,
                                  int32_t ntiles_u, double2* part, const int32_t* tpair,
                                  hipStream_t s, const Ev& ev);
hipError_t launch_lars_rates(const int32_t* tpair, const double2* part, int32_t ntens,
                             double gamma, double eta, double eps, double* rate,
                             double* rate_out, hipStream_t s, const Ev& ev);

}  // namespace tkef

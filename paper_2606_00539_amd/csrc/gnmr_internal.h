// Internal declarations shared by the runtime and the kernels of libgnmr.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gnmr.h"
#include "k1_geometry.h"

namespace gnmr {

// Step counters accumulated by K2 (integer atomics) and read by K3.
enum : int {
  kCntCand = 0,       // |C_t|
  kCntTrigG = 1,      // recoverable units with GNMR / alpha > 1
  kCntTrigD = 2,      // recoverable units with Delta-GNMR / beta > 1
  kCntTrigR = 3,      // recoverable units with R > 1
  kCntNonFinite = 4,  // units with a non-finite norm
  kCntRank = 5,       // members of C_t that are ranked for the budget
  kNumCounters = 8
};

// K2 spreads its counters and candidate list over this many sets (workgroup
// w adds to set w % kCounterSets), so that its global atomics do not queue
// on one address; K3 gathers the sets.
constexpr int kCounterSets = 64;
// Entries per set of the candidate list for U units: a set receives at most
// ceil(workgroups / kCounterSets) workgroups of at most 256 units each.
inline int64_t cand_list_cap(int64_t num_units) { return num_units / kCounterSets + 512; }

// Per-unit flag bits written by K2 and read by K3.
enum : uint8_t {
  kFlagTrigG = 1,      // GNMR / alpha > 1
  kFlagTrigD = 2,      // Delta-GNMR / beta > 1
  kFlagNonFinite = 4,  // non-finite norm
  kFlagTrigR = 8,      // R > 1
  kFlagRec = 16,       // recoverable
  kFlagCand = 32,      // member of the candidate pool C_t
  kFlagKeep = 64       // active without ranking (warm-up; continuing unit under
                       // the admitted-only budget)
};

struct UpdateArgs {
  int32_t num_units;
  int32_t window;      // delta
  int32_t admitted;    // budget_mode == GNMR_BUDGET_ADMITTED
  int32_t static_set;  // budget_mode == GNMR_BUDGET_STATIC
  int32_t warmup;      // warmup_steps (W)
  const int64_t* step; // steps completed so far (device); this step is *step + 1
  double eps, alpha, beta;
  const int64_t* unit_item_off;  // [U+1]
  const float* partial;          // [items]
  const double* ext_norm;        // [U] or nullptr
  double* A;                     // [U]
  double* Q;                     // [window][U]
  double* norm;
  double* gnmr;
  double* dgnmr;
  double* risk;
  const uint8_t* rec;            // [U]
  int32_t* lock;                 // [U], Lock after step t-1 (cleared for units outside C_t)
  uint64_t* keys;                // [U], candidate key or 0
  uint8_t* flags;
  uint8_t* mask;                 // [U], A_{t-1} on entry; cleared for units outside C_t
  int32_t* counters;             // [kCounterSets][kNumCounters], zero on entry
  int32_t* cand_list;            // [kCounterSets][list_cap]: set j holds counters[j][kCntCand]
                                 // members of C_t (any order)
  int64_t list_cap;              // entries per set of cand_list
  double* gsum;                  // [U], sum of GNMR over the static baseline's profiling steps
};

struct SelectArgs {
  int32_t num_units;
  int32_t max_o;
  int32_t lock_len;
  int32_t warmup;      // warmup_steps (W)
  int64_t* step;       // steps completed (device); advanced by one at the end of K3
  const uint8_t* flags;
  const uint64_t* keys;
  int32_t* counters;         // from K2, [num_sets][kNumCounters]; reset to zero for the next step
  const int32_t* cand_list;  // from K2, [num_sets][list_cap]
  int32_t num_sets;          // kCounterSets (one in the single-workgroup kernel)
  int64_t list_cap;
  int32_t* lock;       // in: Lock after step t-1; out: after step t
  uint8_t* mask;
  gnmr_stats* stats;
};

// K4 (actuator): up to kK4Vpt 16-byte vectors per lane; one wavefront per
// row of at most kK4WaveCols bf16 features, one workgroup per longer row of
// at most kK4MaxCols.
constexpr int kK4Block = 256;
constexpr int kK4Vpt = 8;
constexpr int kK4WaveCols = 64 * kK4Vpt * 8;
constexpr int kK4MaxCols = kK4Block * kK4Vpt * 8;
// A launch's grid holds fewer than 2^32 work items: at most this many
// workgroups of kK4Block lanes, i.e. this many wide rows or four times as many
// narrow ones per launch.
constexpr int64_t kK4MaxWorkgroups = int64_t(UINT32_MAX) / kK4Block;

struct ActSeg {
  const char* in;
  char* out;
  int32_t cols;
  int32_t unit;
};
static_assert(sizeof(ActSeg) == 24, "ActSeg layout");

struct RowItem {
  int32_t seg;
  int32_t row;
};

// K5 (weight-gradient GEMM with the sum of squares in its epilogue):
// 256x256 output tiles, K steps of 64, four waves; tiles walked in groups of
// kWgGroupRows tile rows.
constexpr int kWgBM = 256;
constexpr int kWgBN = 256;
constexpr int kWgBK = 64;
constexpr int kWgThreads = 256;
constexpr int kWgGroupRows = 8;

constexpr int kWgMaxBatch = 16;   // problems per launch (passed by value)

struct WgProblem {
  const uint16_t* dy;  // [K][M]
  const uint16_t* x;   // [K][N]
  uint16_t* dw;        // [M][N]
  float* tile_ss;      // [tiles_m * tiles_n]
  int64_t K;
  int32_t M, N, tiles_m, tiles_n;
  int32_t tile_begin;  // first tile of this problem in the launch's tile order
  int32_t accumulate;  // 1: add the product to the stored dw
};

struct WgBatch {
  int32_t num;
  int32_t total_tiles;
  WgProblem p[kWgMaxBatch];
};

int64_t wgrad_tiles(int32_t M, int32_t N);
hipError_t launch_wgrad(const WgBatch& batch, hipStream_t s);
// Rows [0, num_narrow) of `items` have at most kK4WaveCols features (one
// wavefront each), rows [num_narrow, num_rows) more (one workgroup each).
hipError_t launch_actuate(const RowItem* items, int64_t num_narrow, int64_t num_rows,
                          const ActSeg* segs, const uint8_t* mask, int fmt_low, int fmt_rec,
                          hipStream_t s);
// One [rows][sg.cols] matrix, no row table: rows <= 4 * UINT32_MAX when
// sg.cols <= kK4WaveCols, else rows <= UINT32_MAX (one workgroup each).
hipError_t launch_actuate_matrix(const ActSeg& sg, int64_t rows, const uint8_t* mask,
                                 int fmt_low, int fmt_rec, hipStream_t s);
hipError_t launch_sumsq(const Item* items, int64_t num_items, const char* const* seg_base,
                        const int32_t* seg_dtype, float* partial, hipStream_t s);
hipError_t launch_unit_sumsq(const int64_t* unit_item_off, const float* partial,
                             int64_t num_items, int32_t num_units, double* out, hipStream_t s);
hipError_t launch_update(const UpdateArgs& a, int64_t num_items, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
// K2 and K3 as one single-workgroup launch: used when the workload is small
// (at most 1024 units, each summed by one thread, or norms given).
bool single_launch_update_select(const UpdateArgs& a, int64_t num_items);
hipError_t launch_update_select(const UpdateArgs& u, const SelectArgs& s, hipStream_t st);

}  // namespace gnmr

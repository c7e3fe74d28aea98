// internal.h - types and launcher declarations shared by the HIP sources of
// libditango (not part of the public C ABI; see include/ditango.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ditango.h"

namespace ditango {

constexpr int kMaxParts = DITANGO_MAX_PARTITIONS;

// One launch of the fresh-state kernel covers every selected partition.
struct AttnArgs {
  const void* q;            // [B][q_len][H][D]
  const void* k;            // [B][S][H][D]
  const void* v;            // [B][S][H][D]
  void* out_states;         // [P][B][q_len][H][D], state dtype
  float* lse_states;        // [P][B][H][q_len]
  int64_t q_len;
  int64_t S;
  int B, H;
  int n_sel;                // number of selected partitions
  int q_tiles;              // ceil(q_len / rows per workgroup)
  float scale_log2;         // scale * log2(e): exponents are taken base 2
  int64_t kv_begin[kMaxParts];
  int32_t kv_len[kMaxParts];
  int32_t slot[kMaxParts];
  // Tail split (bf16 kernel): logical tasks [n_main, n_main + n_split) run
  // as split_f workgroups each, over consecutive key ranges, writing partial
  // states to part_out / part_lse; a fix-up kernel composes them into the
  // slots.  n_split = 0: every task is one workgroup (n_main is set by the
  // launcher).
  int n_main;
  int n_split;
  int split_f;
  float* part_out;          // [n_split * split_f][rows per workgroup][D]
  float* part_lse;          // [n_split * split_f][rows per workgroup]
  // Balancing over the XCDs (bf16 kernel, with a workspace).  The units of
  // work (main tasks, then split units) are dealt into 8 lists, one per
  // XCD: list x holds the x-th contiguous eighth of the main tasks, then the
  // x-th eighth of the split units.  Workgroups [0, n_static) run fixed
  // units: workgroup b position b / 8 of list b % 8.  Every later workgroup
  // claims one unit from the queue counters of the positions past
  // n_static / 8 (queue x: list x's main tasks, queue 8 + x: its split
  // units): main tasks anywhere before split units, its own XCD's first; it
  // exits when all are exhausted.  queue = null: no queues, every workgroup
  // is static (n_static = n_main, no split units).
  int n_static;
  int* queue;               // kQueueInts counters, zeroed before the launch
};

constexpr int kMaxSplit = 8;
constexpr int kQueueInts = 16;
constexpr size_t kQueueBytes = 256;   // the queue counters, at the start of the workspace

// Tail split plan.  With `slots` workgroups resident at once and `tasks`
// tasks of `tiles` key tiles each, the last round runs rem = tasks % slots
// of them.  Its cost, in key tiles, is estimated as tiles + kMainUnitCost
// unsplit; split into f key ranges it is ceil(f * rem / slots) rounds of
// ceil(tiles / f) + kSplitUnitCost (a split unit loads its queries again and
// writes its partial state in float32), plus kFixupCost for the kernel that
// composes the partials.  Returns the f in [2, kMaxSplit] with the lowest
// estimate (the smallest on ties) when it is at least 3 % below the
// unsplit one, else 1.  Launches with more than kMaxSplitRounds full rounds
// before the last are not split: the workgroups' speeds differ by a few
// percent, so after many rounds their finish times are spread over much of
// a task and the queue counters hand the last tasks to the earliest
// finishers (measured: a 4,440-task launch on 256 CUs ran 0.4-1.2 % faster
// balanced and unsplit than balanced and split 5 or 8 ways, on three
// cards; 1,480 and 8,880 tasks alike; a 216-task single round of 22-tile
// tasks was twice as slow split 7 ways).
constexpr int kMainUnitCost = 1;
constexpr int kSplitUnitCost = 4;
constexpr int kFixupCost = 3;
constexpr int kMaxSplitRounds = 4;

inline int plan_tail_split(int64_t tasks, int64_t slots, int64_t tiles) {
  if (slots <= 0 || tiles <= 0) return 1;
  if (tasks / slots > kMaxSplitRounds) return 1;
  const int64_t rem = tasks % slots;
  if (rem == 0) return 1;
  const double unsplit = (double)(tiles + kMainUnitCost);
  int best = 1;
  double best_t = unsplit;
  for (int f = 2; f <= kMaxSplit; ++f) {
    const int64_t rounds = (f * rem + slots - 1) / slots;
    const double t = (double)(rounds * ((tiles + f - 1) / f + kSplitUnitCost) + kFixupCost);
    if (t < best_t - 1e-9) {
      best_t = t;
      best = f;
    }
  }
  return best_t <= 0.97 * unsplit ? best : 1;
}

struct MergeArgs {
  const void* states;       // [P][rows][D]  (rows = B*q_len*H)
  const float* lse;         // [P][B][H][q_len]
  void* out;                // [rows][D]
  float* lse_out;           // [B][H][q_len] or null
  int64_t q_len;
  int64_t rows;             // B*q_len*H
  int B, H;
  int n;                    // number of listed slots
  int32_t slots[kMaxParts];
};

struct ContribArgs {
  const float* lse;         // [P][n_rows]
  const float* lse_out;     // [n_rows]
  float* w_rows;            // [n_rows][P] or null
  float* w_part;            // [P]
  float* partial;           // workspace [n_blocks][P]
  int64_t n_rows;           // B*H*q_len
  int P;
  int n_blocks;
};

struct NormArgs {
  const void* states;       // [P][elems]
  const void* ref;          // [elems] or null
  float* norms;             // [n]
  float* partial;           // workspace [n][blocks]
  int64_t elems;            // B*q_len*H*D (a multiple of 8)
  int n;
  int blocks;               // workgroups per slot
  int32_t slots[kMaxParts];
};

constexpr int kNormThreads = 256;
constexpr int kNormChunksPerBlock = kNormThreads * 16;   // 8-element chunks per workgroup

// Workgroups of the contrib launch over n_rows rows of the composed-LSE
// array (the workspace holds one partial sum per workgroup and partition).
int64_t contrib_blocks(int64_t n_rows);

// bf16 inputs; states in bf16, or in float32 when state_f32
hipError_t launch_attn_bf16(const AttnArgs& a, int D, bool state_f32, hipStream_t s);
// Bytes of workspace a bf16 launch uses on the current device: the queue
// counters, and the partial states of the tail split when a split shortens
// the last round (0: nothing is launched); `a` needs q_len, B, H and n_sel.
hipError_t attn_bf16_ws_bytes(const AttnArgs& a, int D, size_t* bytes);
// The same launch with a workspace: balanced over the XCDs when `ws_bytes`
// covers the queue counters, and with the tail split as well when it covers
// attn_bf16_ws_bytes; a null workspace runs the static assignment.
hipError_t launch_attn_bf16_ws(const AttnArgs& a, int D, bool state_f32, void* ws, size_t ws_bytes,
                               hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, int D, hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, ditango_dtype sdt, ditango_dtype odt, int D,
                        hipStream_t s);
hipError_t launch_contrib(const ContribArgs& a, hipStream_t s);
// Device address, on the current device, of the fixed scratch array of the
// allocation-free contrib entry point (kContribScratchBytes); looked up once
// per device.
constexpr size_t kContribScratchBytes = DITANGO_CONTRIB_SCRATCH_BYTES;
hipError_t contrib_scratch(float** ptr);
hipError_t launch_norms(const NormArgs& a, ditango_dtype dt, hipStream_t s);

constexpr int kProbeThreads = 256;   // 4 waves per workgroup
hipError_t launch_probe_mfma(int n_workgroups, int iters, float* sink, hipStream_t s);

// Workgroup index remap for the 8 XCDs of the chip: hardware hands out
// consecutive workgroup ids round-robin over the XCDs, so id b runs on XCD
// b % 8.  The remap gives every XCD a contiguous run of logical task ids, so
// tasks that read the same key/value rows (consecutive query tiles of one
// head and partition) share that XCD's L2.
__device__ __forceinline__ int xcd_first(int x, int n) { return x * (n >> 3) + min(x, n & 7); }
__device__ __forceinline__ int xcd_len(int x, int n) { return (n >> 3) + (x < (n & 7) ? 1 : 0); }

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  constexpr int kXcd = 8;
  const int per = nblocks / kXcd;
  const int rem = nblocks % kXcd;
  const int x = bid % kXcd;
  const int i = bid / kXcd;
  return x * per + (x < rem ? x : rem) + i;
}

}  // namespace ditango

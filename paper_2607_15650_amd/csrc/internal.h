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
  // Balancing over the XCDs (bf16 kernel, with a workspace).  The main tasks
  // are cut into 8 contiguous ranges, one per XCD (xcd_first / xcd_len).
  // Workgroups [0, n_static) run fixed tasks: workgroup b the (b / 8)-th
  // task of range b % 8.  Every later workgroup claims one unit from the
  // queue counters: queue x < 8 holds the rest of range x, queue 8 the
  // n_split * split_f split units; its own XCD's queue first, then the main
  // queue with the most left, then the split queue; it exits when all are
  // exhausted.  queue = null: no queues, every workgroup is static
  // (n_static = n_main).
  int n_static;
  int* queue;               // kQueueInts counters, zeroed before the launch
};

constexpr int kMaxSplit = 8;
constexpr int kQueueInts = 16;
constexpr size_t kQueueBytes = 256;   // the queue counters, at the start of the workspace

// Tail split plan: with `slots` workgroups resident at once and `tasks`
// equal-length tasks, the last round runs tasks % slots of them; splitting
// each of those into f key ranges shortens it to ceil(f * rem / slots) / f
// of a task.  Returns the f in [2, kMaxSplit] that minimises that (the
// smallest on ties), or 1 when no split shortens the last round.
inline int plan_tail_split(int64_t tasks, int64_t slots) {
  if (slots <= 0) return 1;
  const int64_t rem = tasks % slots;
  if (rem == 0) return 1;
  int best = 1;
  double best_t = 1.0;
  for (int f = 2; f <= kMaxSplit; ++f) {
    const double t = (double)((f * rem + slots - 1) / slots) / f;
    if (t < best_t - 1e-12) {
      best_t = t;
      best = f;
    }
  }
  return best;
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

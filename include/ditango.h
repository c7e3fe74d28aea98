/*
 * ditango.h - C ABI of the selective attention-state hot path (gfx950).
 *
 * One context-parallel rank's share of one DiT attention call at one
 * denoising step: the rank's query block attends to P key/value partitions of
 * the sequence.  Selected partitions get a fresh attention state, the others
 * keep the state cached at an earlier step, all states are composed, and the
 * contribution weight of every partition is reported for the next step's
 * selection (the paper: Sec. 2.2.4, Eq. attention_state and Eq. composition;
 * Sec. 4.1.2, Eq. lse_weight; Sec. 5.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Device pointers point to device memory (HBM) of the current HIP device;
 *    host pointers (offsets, select, slot lists) are read during the call only.
 *  - The caller allocates every buffer, the contrib workspace included.  The
 *    library allocates nothing, frees nothing and never synchronises: kernels
 *    are enqueued on `stream` (a hipStream_t; NULL = the default stream) and
 *    run asynchronously.  The library keeps no state between calls and may be
 *    called from several host threads.
 *  - Tensors are dense and row-major.  Q is [B][q_len][H][D], K and V are
 *    [B][S][H][D] (batch, sequence, head, head-dim, the layout in which the
 *    paper states its workloads).  An attention state of one partition is an
 *    output OUT [B][q_len][H][D] (normalised, in the state dtype) plus a
 *    log-sum-exp LSE [B][H][q_len] (float32, natural log, includes `scale`).
 *    The state cache is a slot array: OUT slots [P][B][q_len][H][D] and LSE
 *    slots [P][B][H][q_len]; slot j holds partition j's state.
 *  - bf16 tensors hold IEEE bfloat16 bit patterns (uint16).  Arithmetic is
 *    float32 (bf16 MFMA products with float32 accumulation for bf16 inputs).
 *  - Argument errors are detected before anything is launched and return
 *    DITANGO_ERR_INVALID or DITANGO_ERR_UNSUPPORTED; a failed launch returns
 *    DITANGO_ERR_HIP.  Nothing is printed and nothing aborts.
 *  - A partition with no keys has LSE = -inf and OUT = 0 and weight 0.
 */
#ifndef DITANGO_H
#define DITANGO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DITANGO_OK = 0,
  DITANGO_ERR_INVALID = 1,      /* null pointer, bad size, offsets decreasing, ... */
  DITANGO_ERR_UNSUPPORTED = 2,  /* valid but not built: head dim, dtype combination */
  DITANGO_ERR_HIP = 3           /* the HIP runtime reported an error at launch */
} ditango_status;

typedef enum {
  DITANGO_F32 = 0,
  DITANGO_BF16 = 1
} ditango_dtype;

/* Largest number of partitions (slots) one call accepts. */
#define DITANGO_MAX_PARTITIONS 64

/*
 * Fresh attention states of the selected key/value partitions
 * (Sec. 2.2.4, Eq. attention_state; one call covers every selected partition).
 *
 * For every partition j with select[j] != 0, every batch b, head h and query
 * row r, with keys c in [kv_offsets[j], kv_offsets[j+1]):
 *     LSE_j[b][h][r] = log sum_c exp(scale * q[b][r][h] . k[b][c][h])
 *     OUT_j[b][r][h] = sum_c exp(scale * q . k_c - LSE_j) * v[b][c][h]
 * and writes them to slot j of out_states / lse_states.
 *
 *   q, k, v      device; dtype `dt`; Q [B][q_len][H][D], K and V [B][S][H][D]
 *                with S = kv_offsets[P].
 *   dt           DITANGO_BF16 or DITANGO_F32 (inputs, states share it).
 *   D            head dim: 64 or 128; H*D at most 65536
 *                (DITANGO_ERR_UNSUPPORTED beyond).
 *   kv_offsets   host, P+1 int64, kv_offsets[0] = 0, non-decreasing.
 *   select       host, P bytes; non-zero = compute partition j fresh.
 *   scale        softmax scale applied to q.k (normally 1/sqrt(D)); finite
 *                and > 0 (DITANGO_ERR_INVALID otherwise: zero, negative,
 *                inf and NaN are rejected before anything is launched).
 *   out_states   device, [P][B][q_len][H][D] in dtype `dt`.
 *   lse_states   device, [P][B][H][q_len] float32.
 *
 * Slots whose select[j] == 0 are neither read nor written: they keep the state
 * cached at an earlier step, which is the reuse.  Selecting no partition is
 * valid and launches nothing.
 */
ditango_status ditango_attn_partition_states(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, float* lse_states, void* stream);

/*
 * The same with the state dtype chosen separately: bf16 inputs may keep
 * their states in float32 (the states at full precision; the composed
 * output of ditango_merge_states may still be bf16).  `out_states` is
 * [P][B][q_len][H][D] in `state_dt`.  state_dt must equal dt, or be
 * DITANGO_F32 with dt = DITANGO_BF16 (DITANGO_ERR_UNSUPPORTED otherwise).
 * ditango_attn_partition_states(...) is this call with state_dt = dt.
 */
ditango_status ditango_attn_partition_states_ex(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, ditango_dtype state_dt, float* lse_states, void* stream);

/*
 * The same with a workspace that lets the launch balance its work over the
 * XCDs and shorten its last round (the same computation, Sec. 2.2.4, Eq.
 * attention_state; split partial states are composed by Eq. composition).
 * A launch is a set of tasks (query tile x head x batch x selected
 * partition) of which the GPU runs a fixed number at a time.
 *  - Balancing: the first 256 bytes of the workspace hold queue counters
 *    (zeroed by a small kernel on `stream` before a launch that claims any
 *    task).  Most tasks run where the hardware places them; the last ones
 *    are claimed from the counters, so that XCDs that run faster take more
 *    of them.
 *  - Tail split: when the last round is partly filled, the launch has at
 *    most 4 full rounds before it (after more, balancing evens out its
 *    end) and an estimate of the round's cost in key tiles says a split
 *    saves 3 %, its tasks are split into up to 8 key ranges whose partial
 *    states go to the rest of the workspace and are composed into their
 *    slots by a second small kernel.
 *
 *   workspace        device, 256-byte aligned.  NULL or under 256 bytes:
 *                    the static launch of ditango_attn_partition_states_ex;
 *                    at least 256: balanced; at least
 *                    ditango_attn_workspace_bytes(...) for this shape and
 *                    selection on the current device: balanced and split.
 *                    Contents on entry are ignored; on return they are
 *                    scratch.  Calls that overlap on one workspace race.
 *   workspace_bytes  its size.
 *
 * Balancing moves tasks between workgroups, not their arithmetic: a
 * balanced unsplit launch is bitwise the static one.  Split results differ
 * from unsplit ones only by the rounding of the composition; all are
 * deterministic.  fp32 inputs ignore the workspace.
 * DITANGO_ERR_INVALID for a misaligned workspace; otherwise as
 * ditango_attn_partition_states_ex.
 */
ditango_status ditango_attn_partition_states_ws(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, ditango_dtype state_dt, float* lse_states,
    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Workspace bytes ditango_attn_partition_states_ws uses for this launch on
 * the current HIP device: 256 for the queue counters, plus the partial
 * states of the tail split when a split shortens the last round (the
 * compute-unit count and the kernel's occupancy decide).  0 for fp32 inputs,
 * an empty selection or invalid arguments.  Host only, enqueues nothing.
 */
size_t ditango_attn_workspace_bytes(ditango_dtype dt, int B, int H, int D, int64_t q_len,
                                    const int64_t* kv_offsets, int P, const uint8_t* select);

/*
 * Composition of cached and fresh states (Sec. 2.2.4, Eq. composition, n-ary):
 *     M = max_j LSE_j,  LSE = M + log sum_j exp(LSE_j - M),
 *     OUT = sum_j exp(LSE_j - LSE) * OUT_j
 * over the slots listed in `slots` (host, n_slots int32 indices in [0, P));
 * slots == NULL means all P slots in order.  Rows whose listed LSEs are all
 * -inf give OUT = 0, LSE = -inf.  Composing a subset into a spare slot is how a
 * group of states is folded into one cached state.
 *
 *   out_states   device, [P][B][q_len][H][D], dtype `state_dt`.
 *   lse_states   device, [P][B][H][q_len] float32.
 *   out          device, [B][q_len][H][D], dtype `out_dt`.
 *   lse_out      device, [B][H][q_len] float32; may be NULL.
 *   D            head dim: 64 or 128.
 * `out` / `lse_out` may be exactly the first listed slot (same base address,
 * same dtype): the composition then happens in place, which is how adjacent
 * group states are folded into one (each output element is written only
 * after the same element of every listed slot has been read).  Any other
 * overlap with a listed slot is not allowed.
 */
ditango_status ditango_merge_states(
    const void* out_states, const float* lse_states, ditango_dtype state_dt,
    int P, const int32_t* slots, int n_slots,
    int B, int H, int D, int64_t q_len,
    void* out, ditango_dtype out_dt, float* lse_out, void* stream);

/*
 * Bytes of device workspace ditango_contrib needs for these sizes.
 */
size_t ditango_contrib_workspace_bytes(int B, int H, int64_t q_len, int P);

/*
 * Contribution weights of the P partition states to the composed state
 * (Sec. 4.1.1 w_i, Sec. 4.1.2 Eq. lse_weight):
 *     W[b][h][r][j] = exp(LSE_j[b][h][r] - LSE[b][h][r])     (0 where LSE = -inf)
 *     w_part[j]     = mean of W[.][.][.][j] over all B*H*q_len rows.
 * The row means are reduced in a fixed order, so results are bitwise
 * identical from run to run.
 *
 *   lse_states   device, [P][B][H][q_len] float32.
 *   lse_out      device, [B][H][q_len] float32 (the composed LSE).
 *   w_rows       device, [B][H][q_len][P] float32, or NULL to skip.
 *   w_part       device, [P] float32.
 *   workspace    device, ditango_contrib_workspace_bytes(...) bytes, 16-byte
 *                aligned; its contents on entry do not matter.
 */
ditango_status ditango_contrib(
    const float* lse_states, const float* lse_out, int P,
    int B, int H, int64_t q_len,
    float* w_rows, float* w_part, void* workspace, void* stream);

/* Size of the fixed device scratch array of ditango_contrib_noalloc. */
#define DITANGO_CONTRIB_SCRATCH_BYTES (1u << 20)

/*
 * ditango_contrib without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same arguments (minus the workspace),
 * same kernels and results bit for bit as ditango_contrib.  Allocates
 * nothing: the per-workgroup partial sums go to a fixed device array of
 * DITANGO_CONTRIB_SCRATCH_BYTES bytes (one per GPU, held until the process
 * ends; its address is looked up on a device's first call).
 *
 * Limit: ditango_contrib_workspace_bytes(B, H, q_len, P) must not exceed
 * DITANGO_CONTRIB_SCRATCH_BYTES (e.g. up to about 16.7 million rows
 * B*H*q_len at P = 8, 2.1 million at P = 64); larger sizes return
 * DITANGO_ERR_UNSUPPORTED before anything is launched.  Every call on one GPU
 * shares that array: calls that overlap on one GPU (on different streams or
 * from several threads) race.  Nothing in the array needs to start at zero:
 * every partial sum a call reads is written earlier in the same call.
 */
ditango_status ditango_contrib_noalloc(
    const float* lse_states, const float* lse_out, int P,
    int B, int H, int64_t q_len,
    float* w_rows, float* w_part, void* stream);

/*
 * Bytes of device workspace ditango_state_norms needs for these sizes.
 */
size_t ditango_norms_workspace_bytes(int B, int H, int D, int64_t q_len, int n_slots);

/*
 * Frobenius norms of state outputs, the quantities of the selection
 * planner's error model (Sec. 4.1.2: the scale ratio alpha(i) =
 * ||AS(i)|| / ||AS(i_loc)||, Eq. scale_ratio, and the local-state drift that
 * Eq. error_extrapolation scales by it):
 *     norms[i] = sqrt( sum over (b, r, h, d) of (OUT_{slots[i]} - REF)^2 )
 * with REF = 0 when `ref` is NULL.  Reduced in a fixed order: bitwise
 * identical from run to run.
 *
 *   out_states   device, [P][B][q_len][H][D], dtype `dt`.
 *   slots        host, n_slots int32 indices in [0, P); NULL = all P slots.
 *   ref          device, [B][q_len][H][D] in dtype `dt`, or NULL.
 *   norms        device, [n_slots] float32.
 *   workspace    device, ditango_norms_workspace_bytes(...) bytes, 16-byte
 *                aligned; its contents on entry do not matter.
 */
ditango_status ditango_state_norms(
    const void* out_states, ditango_dtype dt, int P, const int32_t* slots, int n_slots,
    int B, int H, int D, int64_t q_len, const void* ref,
    float* norms, void* workspace, void* stream);

/*
 * Device characterisation, not part of the method: the dense bf16 MFMA rate
 * the GPU sustains at the clock it runs at under MFMA load, to hold the
 * attention kernel against beside the published peak.  Launches
 * n_workgroups workgroups of 256 threads (4 waves); every wave issues `iters`
 * rounds of four independent 32x32x16 bf16 MFMAs and nothing else, so one
 * call performs n_workgroups * 4 * iters * 4 * 32768 flops.  Time it with
 * events on `stream`.
 *
 *   n_workgroups  1 .. 1048576 (use several per compute unit).
 *   iters         1 .. 1048576.
 *   sink          device, n_workgroups * 256 float32; receives one value per
 *                 thread that keeps the products live (meaningless otherwise).
 */
ditango_status ditango_probe_mfma_bf16(int n_workgroups, int iters, float* sink, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* ditango_status_string(ditango_status s);

/* Library version as "major.minor.patch". */
const char* ditango_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DITANGO_H */

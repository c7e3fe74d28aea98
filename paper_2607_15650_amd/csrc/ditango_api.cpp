// ditango_api.cpp - the C ABI of libditango: argument validation and launches.
// Every check happens on the host before anything is enqueued; the kernels
// live in attn_bf16.hip, attn_f32.hip and merge.hip.
#include <math.h>
#include <string.h>

#include "internal.h"

using namespace ditango;

namespace {

bool valid_dtype(ditango_dtype d) { return d == DITANGO_F32 || d == DITANGO_BF16; }

ditango_status from_hip(hipError_t e) { return e == hipSuccess ? DITANGO_OK : DITANGO_ERR_HIP; }

}  // namespace

extern "C" {

const char* ditango_status_string(ditango_status s) {
  switch (s) {
    case DITANGO_OK: return "ok";
    case DITANGO_ERR_INVALID: return "invalid argument";
    case DITANGO_ERR_UNSUPPORTED: return "unsupported configuration";
    case DITANGO_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* ditango_version(void) { return "0.1.0"; }

}  // extern "C"

namespace {

// Argument checks shared by the attention entry points; fills `a` (not the
// launch fields).  Returns DITANGO_OK when a launch may proceed.
ditango_status attn_args(const void* q, const void* k, const void* v, ditango_dtype dt, int B, int H, int D,
                         int64_t q_len, const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
                         const void* out_states, ditango_dtype state_dt, const float* lse_states, AttnArgs* a) {
  if (!q || !k || !v || !kv_offsets || !select || !out_states || !lse_states) return DITANGO_ERR_INVALID;
  if (!valid_dtype(dt) || !valid_dtype(state_dt)) return DITANGO_ERR_INVALID;
  if (state_dt != dt && !(dt == DITANGO_BF16 && state_dt == DITANGO_F32)) return DITANGO_ERR_UNSUPPORTED;
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return DITANGO_ERR_INVALID;
  if (P > kMaxParts) return DITANGO_ERR_UNSUPPORTED;
  if (D != 64 && D != 128) return DITANGO_ERR_UNSUPPORTED;
  // the kernels mask keys past a partition's end to -inf before scaling and
  // take the running maximum of the unscaled scores: both need scale > 0
  if (!isfinite(scale) || !(scale > 0.f)) return DITANGO_ERR_INVALID;
  if (kv_offsets[0] != 0) return DITANGO_ERR_INVALID;
  for (int j = 0; j < P; ++j) {
    if (kv_offsets[j + 1] < kv_offsets[j]) return DITANGO_ERR_INVALID;
    if (kv_offsets[j + 1] - kv_offsets[j] > 0x7fffffffLL) return DITANGO_ERR_UNSUPPORTED;
  }
  // row indices of a query tile and element offsets stay in int64; the
  // per-partition key count must fit int32 (checked above), so must q_len.
  if (q_len > 0x7fffffffLL) return DITANGO_ERR_UNSUPPORTED;
  // the bf16 kernel addresses a key tile with 32-bit lane offsets from its
  // first row: H*D <= 65536 keeps a tile of up to 128 keys within 16 MiB
  if ((int64_t)H * D > 65536) return DITANGO_ERR_UNSUPPORTED;

  memset(a, 0, sizeof(*a));
  a->q = q;
  a->k = k;
  a->v = v;
  a->out_states = const_cast<void*>(out_states);
  a->lse_states = const_cast<float*>(lse_states);
  a->q_len = q_len;
  a->S = kv_offsets[P];
  a->B = B;
  a->H = H;
  a->scale_log2 = scale * 1.4426950408889634f;
  int n = 0;
  for (int j = 0; j < P; ++j) {
    if (!select[j]) continue;
    a->kv_begin[n] = kv_offsets[j];
    a->kv_len[n] = (int32_t)(kv_offsets[j + 1] - kv_offsets[j]);
    a->slot[n] = j;
    ++n;
  }
  a->n_sel = n;
  return DITANGO_OK;
}

}  // namespace

extern "C" {

ditango_status ditango_attn_partition_states_ws(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, ditango_dtype state_dt, float* lse_states,
    void* workspace, size_t workspace_bytes, void* stream) {
  AttnArgs a;
  const ditango_status st = attn_args(q, k, v, dt, B, H, D, q_len, kv_offsets, P, select, scale, out_states,
                                      state_dt, lse_states, &a);
  if (st != DITANGO_OK) return st;
  if (workspace != nullptr && ((uintptr_t)workspace & 255u) != 0) return DITANGO_ERR_INVALID;
  if (a.n_sel == 0) return DITANGO_OK;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DITANGO_BF16)
    return from_hip(launch_attn_bf16_ws(a, D, state_dt == DITANGO_F32, workspace_bytes > 0 ? workspace : nullptr,
                                        workspace_bytes, s));
  return from_hip(launch_attn_f32(a, D, s));
}

ditango_status ditango_attn_partition_states_ex(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, ditango_dtype state_dt, float* lse_states, void* stream) {
  return ditango_attn_partition_states_ws(q, k, v, dt, B, H, D, q_len, kv_offsets, P, select, scale, out_states,
                                          state_dt, lse_states, nullptr, 0, stream);
}

size_t ditango_attn_workspace_bytes(ditango_dtype dt, int B, int H, int D, int64_t q_len,
                                    const int64_t* kv_offsets, int P, const uint8_t* select) {
  if (dt != DITANGO_BF16) return 0;
  // placeholders stand in for the tensors: only the shape and the selection
  // decide the plan
  static const char dummy[4] = {0};
  AttnArgs a;
  if (attn_args(dummy, dummy, dummy, dt, B, H, D, q_len, kv_offsets, P, select, 1.0f, dummy, dt,
                (const float*)dummy, &a) != DITANGO_OK || a.n_sel == 0)
    return 0;
  size_t bytes = 0;
  if (attn_bf16_ws_bytes(a, D, &bytes) != hipSuccess) return 0;
  return bytes;
}

ditango_status ditango_attn_partition_states(
    const void* q, const void* k, const void* v, ditango_dtype dt,
    int B, int H, int D, int64_t q_len,
    const int64_t* kv_offsets, int P, const uint8_t* select, float scale,
    void* out_states, float* lse_states, void* stream) {
  return ditango_attn_partition_states_ex(q, k, v, dt, B, H, D, q_len, kv_offsets, P, select, scale,
                                          out_states, dt, lse_states, stream);
}

ditango_status ditango_merge_states(
    const void* out_states, const float* lse_states, ditango_dtype state_dt,
    int P, const int32_t* slots, int n_slots,
    int B, int H, int D, int64_t q_len,
    void* out, ditango_dtype out_dt, float* lse_out, void* stream) {
  if (!out_states || !lse_states || !out) return DITANGO_ERR_INVALID;
  if (!valid_dtype(state_dt) || !valid_dtype(out_dt)) return DITANGO_ERR_INVALID;
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return DITANGO_ERR_INVALID;
  if (P > kMaxParts) return DITANGO_ERR_UNSUPPORTED;
  if (D != 64 && D != 128) return DITANGO_ERR_UNSUPPORTED;
  MergeArgs a;
  memset(&a, 0, sizeof(a));
  if (slots == nullptr) {
    n_slots = P;
    for (int j = 0; j < P; ++j) a.slots[j] = j;
  } else {
    if (n_slots < 1 || n_slots > kMaxParts) return DITANGO_ERR_INVALID;
    for (int j = 0; j < n_slots; ++j) {
      if (slots[j] < 0 || slots[j] >= P) return DITANGO_ERR_INVALID;
      a.slots[j] = slots[j];
    }
  }
  a.states = out_states;
  a.lse = lse_states;
  a.out = out;
  a.lse_out = lse_out;
  a.q_len = q_len;
  a.rows = (int64_t)B * q_len * H;
  a.B = B;
  a.H = H;
  a.n = n_slots;
  return from_hip(launch_merge(a, state_dt, out_dt, D, (hipStream_t)stream));
}

size_t ditango_contrib_workspace_bytes(int B, int H, int64_t q_len, int P) {
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return 0;
  const int64_t n_rows = (int64_t)B * H * q_len;
  return (size_t)(contrib_blocks(n_rows) * P * (int64_t)sizeof(float));
}

ditango_status ditango_contrib(
    const float* lse_states, const float* lse_out, int P,
    int B, int H, int64_t q_len,
    float* w_rows, float* w_part, void* workspace, void* stream) {
  if (!lse_states || !lse_out || !w_part || !workspace) return DITANGO_ERR_INVALID;
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return DITANGO_ERR_INVALID;
  if (P > kMaxParts) return DITANGO_ERR_UNSUPPORTED;
  if (((uintptr_t)workspace & 15u) != 0) return DITANGO_ERR_INVALID;
  ContribArgs a;
  memset(&a, 0, sizeof(a));
  a.lse = lse_states;
  a.lse_out = lse_out;
  a.w_rows = w_rows;
  a.w_part = w_part;
  a.partial = (float*)workspace;
  a.n_rows = (int64_t)B * H * q_len;
  a.P = P;
  const int64_t nb = contrib_blocks(a.n_rows);
  if (nb > 0x7fffffffLL) return DITANGO_ERR_UNSUPPORTED;
  a.n_blocks = (int)nb;
  return from_hip(launch_contrib(a, (hipStream_t)stream));
}

ditango_status ditango_contrib_noalloc(
    const float* lse_states, const float* lse_out, int P,
    int B, int H, int64_t q_len,
    float* w_rows, float* w_part, void* stream) {
  if (!lse_states || !lse_out || !w_part) return DITANGO_ERR_INVALID;
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return DITANGO_ERR_INVALID;
  if (P > kMaxParts) return DITANGO_ERR_UNSUPPORTED;
  // the partial sums must fit the fixed scratch array
  if (ditango_contrib_workspace_bytes(B, H, q_len, P) > kContribScratchBytes) return DITANGO_ERR_UNSUPPORTED;
  float* partial = nullptr;
  if (contrib_scratch(&partial) != hipSuccess) return DITANGO_ERR_HIP;
  ContribArgs a;
  memset(&a, 0, sizeof(a));
  a.lse = lse_states;
  a.lse_out = lse_out;
  a.w_rows = w_rows;
  a.w_part = w_part;
  a.partial = partial;
  a.n_rows = (int64_t)B * H * q_len;
  a.P = P;
  a.n_blocks = (int)contrib_blocks(a.n_rows);
  return from_hip(launch_contrib(a, (hipStream_t)stream));
}

static int64_t norm_blocks(int B, int H, int D, int64_t q_len) {
  const int64_t chunks = (int64_t)B * q_len * H * D / 8;
  return (chunks + kNormChunksPerBlock - 1) / kNormChunksPerBlock;
}

size_t ditango_norms_workspace_bytes(int B, int H, int D, int64_t q_len, int n_slots) {
  if (B < 1 || H < 1 || q_len < 1 || n_slots < 1 || (D != 64 && D != 128)) return 0;
  return (size_t)(norm_blocks(B, H, D, q_len) * n_slots * (int64_t)sizeof(float));
}

ditango_status ditango_state_norms(
    const void* out_states, ditango_dtype dt, int P, const int32_t* slots, int n_slots,
    int B, int H, int D, int64_t q_len, const void* ref,
    float* norms, void* workspace, void* stream) {
  if (!out_states || !norms || !workspace) return DITANGO_ERR_INVALID;
  if (!valid_dtype(dt)) return DITANGO_ERR_INVALID;
  if (B < 1 || H < 1 || q_len < 1 || P < 1) return DITANGO_ERR_INVALID;
  if (P > kMaxParts) return DITANGO_ERR_UNSUPPORTED;
  if (D != 64 && D != 128) return DITANGO_ERR_UNSUPPORTED;
  if (((uintptr_t)workspace & 15u) != 0) return DITANGO_ERR_INVALID;
  NormArgs a;
  memset(&a, 0, sizeof(a));
  if (slots == nullptr) {
    n_slots = P;
    for (int j = 0; j < P; ++j) a.slots[j] = j;
  } else {
    if (n_slots < 1 || n_slots > kMaxParts) return DITANGO_ERR_INVALID;
    for (int j = 0; j < n_slots; ++j) {
      if (slots[j] < 0 || slots[j] >= P) return DITANGO_ERR_INVALID;
      a.slots[j] = slots[j];
    }
  }
  const int64_t nb = norm_blocks(B, H, D, q_len);
  if (nb > 0x7fffffffLL) return DITANGO_ERR_UNSUPPORTED;
  a.states = out_states;
  a.ref = ref;
  a.norms = norms;
  a.partial = (float*)workspace;
  a.elems = (int64_t)B * q_len * H * D;
  a.n = n_slots;
  a.blocks = (int)nb;
  return from_hip(launch_norms(a, dt, (hipStream_t)stream));
}

ditango_status ditango_probe_mfma_bf16(int n_workgroups, int iters, float* sink, void* stream) {
  if (!sink || n_workgroups < 1 || iters < 1) return DITANGO_ERR_INVALID;
  if (n_workgroups > (1 << 20) || iters > (1 << 20)) return DITANGO_ERR_INVALID;
  return from_hip(launch_probe_mfma(n_workgroups, iters, sink, (hipStream_t)stream));
}

}  // extern "C"

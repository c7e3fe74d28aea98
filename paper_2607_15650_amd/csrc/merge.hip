// merge.hip - composition of attention states and contribution weights (gfx950).
//
// merge: the n-ary state composition of Sec. 2.2.4 (Eq. composition),
//   M = max_j LSE_j, LSE = M + log sum_j e^{LSE_j - M}, OUT = sum_j e^{LSE_j - LSE} OUT_j,
// over a list of cached/fresh state slots.  Pure streaming: every OUT slot is
// read once and the output written once, so the kernel is bound by HBM
// bandwidth.  A row's LSE loads are issued first, then its state loads; the
// weights are formed while the states are in flight.
//
// contrib: per-row weights W_j = e^{LSE_j - LSE} (w_i of Sec. 4.1.1; the
// anchor weights of Eq. lse_weight) and their mean over all rows per
// partition, reduced in a fixed order (workgroup tree, then one workgroup over
// the per-workgroup partial sums) so results are bitwise reproducible.
#include <mutex>

#include "internal.h"

namespace ditango {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 8 consecutive elements of a state row: loaded in the state type (bf16
// chunks stay 4 registers until they are weighted), used as float
template <typename T> struct Chunk8;
template <> struct Chunk8<__bf16> {
  typedef bf16x8 type;
  static __device__ __forceinline__ type load(const __bf16* p) { return __builtin_nontemporal_load((const bf16x8*)p); }
  static __device__ __forceinline__ f32x8 f32(const type& x) { return __builtin_convertvector(x, f32x8); }
  static __device__ __forceinline__ void store(__bf16* p, const f32x8& v) {
    __builtin_nontemporal_store(__builtin_convertvector(v, bf16x8), (bf16x8*)p);
  }
};
template <> struct Chunk8<float> {
  typedef f32x8 type;
  static __device__ __forceinline__ type load(const float* p) {
    const f32x4 a = __builtin_nontemporal_load((const f32x4*)p);
    const f32x4 b = __builtin_nontemporal_load((const f32x4*)(p + 4));
    return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
  static __device__ __forceinline__ f32x8 f32(const type& x) { return x; }
  static __device__ __forceinline__ void store(float* p, const f32x8& v) {
    __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, (f32x4*)p);
    __builtin_nontemporal_store(f32x4{v[4], v[5], v[6], v[7]}, (f32x4*)(p + 4));
  }
};

constexpr int kMergeThreads = 64;      // small workgroups keep every CU evenly fed
constexpr int kMergeBatch = 8;         // slots whose loads are in flight together

// Each thread owns one 8-element chunk of one row (row = (b*q_len + r)*H + h,
// rows contiguous in every slot), so the CPR = D/8 lanes of a row are
// consecutive lanes of one wave.  The thread first issues the loads of the
// row's LSEs (the row's lanes share the addresses, so each load instruction
// touches one line per row), then the state loads of the first batch of
// slots; it forms the row's maximum, log-sum-exp and weights itself (no
// cross-lane exchange, no LDS, no barrier) while the states are in flight,
// and weights each chunk as it lands: OUT = sum_j w_j OUT_j in float32.
// Issuing the LSE loads first makes the weights ready before the first chunk
// arrives, so no chunk waits in registers for them (measured at the
// video-DiT shape: 148.7 / 156.6 us warm / cold against 152.6 / 159.5 us
// with the state loads first).
// NMAX bounds the slot count n (read from the arguments): every loop is
// unrolled over NMAX with wave-uniform guards, so the weights stay in
// registers and small counts (group composition: 2 slots; a composed step:
// a handful) use a small, high-occupancy instantiation.  IDX32: row and LSE
// indices in 32-bit arithmetic (a 64-bit division by a run-time value is a
// long instruction sequence in front of the LSE loads).
template <typename TS, typename TO, int D, int NMAX, bool IDX32>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const MergeArgs a) {
  constexpr int CPR = D / 8;                      // chunks (lanes) per row
  using CK = Chunk8<TS>;
  const int n = a.n;
  const int64_t c = (int64_t)blockIdx.x * kMergeThreads + threadIdx.x;
  const bool live = c < a.rows * CPR;
  const int64_t row = live ? c / CPR : 0;
  const int ch = (int)(c % CPR);
  const int64_t slot_elems = a.rows * D;
  const int64_t lse_slot = (int64_t)a.B * a.H * a.q_len;
  const TS* __restrict__ st = (const TS*)a.states + row * D + ch * 8;

  // LSE index of the row: (b*H + h)*q_len + r for row = (b*q_len + r)*H + h
  int64_t li;
  if constexpr (IDX32) {
    const uint32_t r32 = (uint32_t)row, H = (uint32_t)a.H, L = (uint32_t)a.q_len;
    const uint32_t br = r32 / H;
    const uint32_t b = br / L;
    li = (int64_t)((b * H + (r32 - br * H)) * L + (br - b * L));
  } else {
    const int h = (int)(row % a.H);
    const int64_t br = row / a.H;
    li = ((br / a.q_len) * a.H + h) * a.q_len + br % a.q_len;
  }
  // Every load is unconditional (a lane past the last row reads row 0, a
  // position past the list reads its first slot): a load under a per-lane
  // condition is issued inside a branch and waited for before the branch
  // ends, which serialises the slots' loads of a thread.
  int sl[NMAX];
#pragma unroll
  for (int j = 0; j < NMAX; ++j) sl[j] = a.slots[j < n ? j : 0];
  float lv[NMAX];
#pragma unroll
  for (int j = 0; j < NMAX; ++j) lv[j] = a.lse[(int64_t)sl[j] * lse_slot + li];
  typename CK::type x[kMergeBatch];
#pragma unroll
  for (int u = 0; u < kMergeBatch && u < NMAX; ++u) x[u] = CK::load(st + (int64_t)sl[u] * slot_elems);
  // (the host guarantees n >= 1: the first position is always listed)
#pragma unroll
  for (int j = 1; j < NMAX; ++j) lv[j] = j < n ? lv[j] : -INFINITY;

  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NMAX; ++j) mx = fmaxf(mx, lv[j]);
  float tot = 0.f;
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    lv[j] = mx == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((lv[j] - mx) * kLog2e);
    tot += lv[j];
  }
  const float inv = tot > 0.f ? 1.0f / tot : 0.f;
  const float lse = tot > 0.f ? mx + __builtin_amdgcn_logf(tot) * kLn2 : -INFINITY;
  auto weight = [&](int j) { return lv[j] * inv; };
  f32x8 acc = f32x8{};
#pragma unroll
  for (int u = 0; u < kMergeBatch && u < NMAX; ++u)
    if (u < n) acc += weight(u) * CK::f32(x[u]);
  // later batches: fully unrolled over the largest slot count so that every
  // weight index is a compile-time constant (the weights stay in registers)
#pragma unroll
  for (int j0 = kMergeBatch; j0 < NMAX; j0 += kMergeBatch) {
    if (j0 < n) {
#pragma unroll
      for (int u = 0; u < kMergeBatch; ++u) x[u] = CK::load(st + (int64_t)sl[j0 + u] * slot_elems);
#pragma unroll
      for (int u = 0; u < kMergeBatch; ++u)
        if (j0 + u < n) acc += weight(j0 + u) * CK::f32(x[u]);
    }
  }
  if (live) {
    Chunk8<TO>::store((TO*)a.out + row * D + ch * 8, acc);
    if (a.lse_out != nullptr && ch == 0) a.lse_out[li] = lse;
  }
}

template <typename TS, typename TO, int D, bool IDX32>
void launch_merge_n(const MergeArgs& a, dim3 g, dim3 t, hipStream_t s) {
  if (a.n <= 4)
    hipLaunchKernelGGL((merge_kernel<TS, TO, D, 4, IDX32>), g, t, 0, s, a);
  else if (a.n <= 8)
    hipLaunchKernelGGL((merge_kernel<TS, TO, D, 8, IDX32>), g, t, 0, s, a);
  else if (a.n <= 16)
    hipLaunchKernelGGL((merge_kernel<TS, TO, D, 16, IDX32>), g, t, 0, s, a);
  else
    hipLaunchKernelGGL((merge_kernel<TS, TO, D, kMaxParts, IDX32>), g, t, 0, s, a);
}

template <typename TS, typename TO, int D>
hipError_t launch_merge_t(const MergeArgs& a, hipStream_t s) {
  const int64_t blocks = (a.rows * (D / 8) + kMergeThreads - 1) / kMergeThreads;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  const dim3 g((unsigned)blocks), t(kMergeThreads);
  if (a.rows < 0x7fffffffLL && (int64_t)a.B * a.H * a.q_len < 0x7fffffffLL)
    launch_merge_n<TS, TO, D, true>(a, g, t, s);
  else
    launch_merge_n<TS, TO, D, false>(a, g, t, s);
  return hipGetLastError();
}

template <typename TS, typename TO>
hipError_t launch_merge_d(const MergeArgs& a, int D, hipStream_t s) {
  if (D == 128) return launch_merge_t<TS, TO, 128>(a, s);
  if (D == 64) return launch_merge_t<TS, TO, 64>(a, s);
  return hipErrorInvalidValue;
}

// ---- contribution weights: per-workgroup partial sums, fixed order
//
// Every thread forms the weights of its rows for all listed partitions at
// once (P accumulators in registers), then each partition's sum is reduced
// with a butterfly over the wave (lane l adds lane l^k's value, so every lane
// holds the same bits) and the waves' sums are added in wave order: one
// barrier for all partitions, and bitwise the same result on every run.
constexpr int kContribThreads = 256;
constexpr int kContribRowsPerThread = 2;
constexpr int kContribRowsPerBlock = kContribThreads * kContribRowsPerThread;
constexpr int kContribWaves = kContribThreads / 64;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int k = 32; k > 0; k >>= 1) x += __shfl_xor(x, k, 64);
  return x;
}

template <int PMAX>
__global__ __launch_bounds__(kContribThreads) void contrib_partial_kernel(const ContribArgs a) {
  constexpr int R = kContribRowsPerThread;
  __shared__ float red[kContribWaves][PMAX];
  const int tid = threadIdx.x;
  const int P = a.P;
  const int64_t n = a.n_rows;
  const float* __restrict__ lse = a.lse;
  const float* __restrict__ lse_out = a.lse_out;
  float* __restrict__ w_rows = a.w_rows;
  const int64_t base = (int64_t)blockIdx.x * kContribRowsPerBlock;
  // every load of the thread's rows first, then the weights: the loads are
  // all in flight at once.  They are unconditional (a row past the end reads
  // the last row, a partition past P reads partition 0; both are masked
  // afterwards): a load under a per-lane condition is waited for inside its
  // branch, one after another.
  float lo[R], lj[R][PMAX];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int64_t r = base + i * kContribThreads + tid;
    const int64_t rc = r < n ? r : n - 1;
    lo[i] = lse_out[rc];
#pragma unroll
    for (int j = 0; j < PMAX; ++j) lj[i][j] = lse[(int64_t)(j < P ? j : 0) * n + rc];
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const bool ok = base + i * kContribThreads + tid < n;
    lo[i] = ok ? lo[i] : -INFINITY;
#pragma unroll
    for (int j = 0; j < PMAX; ++j) lj[i][j] = (ok && j < P) ? lj[i][j] : -INFINITY;
  }
  float acc[PMAX];
#pragma unroll
  for (int j = 0; j < PMAX; ++j) acc[j] = 0.f;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int64_t r = base + i * kContribThreads + tid;
#pragma unroll
    for (int j = 0; j < PMAX; ++j) {
      if (j < P) {
        float w = 0.f;
        if (lo[i] != -INFINITY && lj[i][j] != -INFINITY) w = __builtin_amdgcn_exp2f((lj[i][j] - lo[i]) * kLog2e);
        if (w_rows != nullptr && r < n) w_rows[r * P + j] = w;
        acc[j] += w;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < PMAX; ++j)
    if (j < P) acc[j] = wave_sum(acc[j]);
  if ((tid & 63) == 0) {
#pragma unroll
    for (int j = 0; j < PMAX; ++j)
      if (j < P) red[tid >> 6][j] = acc[j];
  }
  __syncthreads();
  if (tid < P) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kContribWaves; ++w) sum += red[w][tid];
    a.partial[(int64_t)blockIdx.x * P + tid] = sum;
  }
}

// The workgroups' partial sums added in a fixed order by one wide workgroup
// (its thread t takes partials t, t + kFinalThreads, ...).
constexpr int kFinalThreads = 1024;
constexpr int kFinalWaves = kFinalThreads / 64;

template <int PMAX>
__global__ __launch_bounds__(kFinalThreads) void contrib_final_kernel(const ContribArgs a) {
  __shared__ float red[kFinalWaves][PMAX];
  const int tid = threadIdx.x;
  const int P = a.P;
  float acc[PMAX];
#pragma unroll
  for (int j = 0; j < PMAX; ++j) acc[j] = 0.f;
  for (int blk = tid; blk < a.n_blocks; blk += kFinalThreads) {
#pragma unroll
    for (int j = 0; j < PMAX; ++j)
      if (j < P) acc[j] += a.partial[(int64_t)blk * P + j];
  }
#pragma unroll
  for (int j = 0; j < PMAX; ++j)
    if (j < P) acc[j] = wave_sum(acc[j]);
  if ((tid & 63) == 0) {
#pragma unroll
    for (int j = 0; j < PMAX; ++j)
      if (j < P) red[tid >> 6][j] = acc[j];
  }
  __syncthreads();
  if (tid < P) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kFinalWaves; ++w) sum += red[w][tid];
    a.w_part[tid] = a.n_rows > 0 ? sum / (float)a.n_rows : 0.f;
  }
}

template <int PMAX>
hipError_t launch_contrib_t(const ContribArgs& a, hipStream_t s) {
  if (a.n_blocks > 0) {
    hipLaunchKernelGGL(contrib_partial_kernel<PMAX>, dim3(a.n_blocks), dim3(kContribThreads), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(contrib_final_kernel<PMAX>, dim3(1), dim3(kFinalThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, ditango_dtype sdt, ditango_dtype odt, int D, hipStream_t s) {
  if (sdt == DITANGO_BF16 && odt == DITANGO_BF16) return launch_merge_d<__bf16, __bf16>(a, D, s);
  if (sdt == DITANGO_BF16 && odt == DITANGO_F32) return launch_merge_d<__bf16, float>(a, D, s);
  if (sdt == DITANGO_F32 && odt == DITANGO_F32) return launch_merge_d<float, float>(a, D, s);
  if (sdt == DITANGO_F32 && odt == DITANGO_BF16) return launch_merge_d<float, __bf16>(a, D, s);
  return hipErrorInvalidValue;
}

int64_t contrib_blocks(int64_t n_rows) { return (n_rows + kContribRowsPerBlock - 1) / kContribRowsPerBlock; }

hipError_t launch_contrib(const ContribArgs& a, hipStream_t s) {
  if (a.P <= 8) return launch_contrib_t<8>(a, s);
  if (a.P <= 16) return launch_contrib_t<16>(a, s);
  return launch_contrib_t<kMaxParts>(a, s);
}

// ---- scratch of the allocation-free contrib entry point
//
// The per-workgroup partial sums live in a file-scope device array: one copy
// per GPU, held until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory, so its device address is looked up
// once per device (with that device current) and only that address is
// passed to kernels.
static __device__ __align__(256) float scratch[kContribScratchBytes / sizeof(float)];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};
}  // namespace

hipError_t contrib_scratch(float** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = (float*)g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace ditango

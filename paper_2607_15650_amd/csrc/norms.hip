// norms.hip - Frobenius norms of attention-state outputs (gfx950).
//
// For listed slots j: || OUT_j - REF ||_2 over all (b, r, h, d), REF optional.
// These feed the error model of the selection planner: the scale ratio
// alpha(i) = ||AS(i)|| / ||AS(i_loc)|| (Sec. 4.1.2, Eq. scale_ratio) and the
// local-state drift ||AS_t(i_loc) - AS_tc(i_loc)|| that the age penalty
// extrapolates (Eq. error_extrapolation).  Bound by HBM: every listed slot
// (and REF once per slot) is read once.  The sums of squares are reduced in a
// fixed order (per-workgroup tree, then one workgroup over the partials), so
// the result is bitwise reproducible.
#include "internal.h"

namespace ditango {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

// 8 consecutive elements, loaded in the state type and used as float
template <typename T> struct Raw8;
template <> struct Raw8<__bf16> {
  typedef bf16x8 type;
  static __device__ __forceinline__ type load(const __bf16* p) { return __builtin_nontemporal_load((const bf16x8*)p); }
  static __device__ __forceinline__ f32x8 f32(const type& x) { return __builtin_convertvector(x, f32x8); }
};
template <> struct Raw8<float> {
  typedef f32x8 type;
  static __device__ __forceinline__ type load(const float* p) {
    const f32x4 a = __builtin_nontemporal_load((const f32x4*)p);
    const f32x4 b = __builtin_nontemporal_load((const f32x4*)(p + 4));
    return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
  static __device__ __forceinline__ f32x8 f32(const type& x) { return x; }
};


// grid: (blocks per slot, n_slots).  Each workgroup sums the squares of a fixed
// range of 8-element chunks of one slot into partial[slot][block].
template <typename T>
__global__ __launch_bounds__(kNormThreads) void norms_partial_kernel(const NormArgs a) {
  __shared__ float red[kNormThreads];
  const int tid = threadIdx.x;
  const int si = blockIdx.y;
  const T* __restrict__ src = (const T*)a.states + (int64_t)a.slots[si] * a.elems;
  const T* __restrict__ ref = (const T*)a.ref;
  const int64_t chunks = a.elems / 8;
  const int64_t c0 = (int64_t)blockIdx.x * kNormChunksPerBlock;
  // batches of kBatch chunks: every load of a batch (state and reference)
  // is issued before the first is used, and unconditionally (a chunk past
  // the end reads the last chunk and is then replaced by zeros, which leave
  // the sum's bits alone): a load under a per-lane condition is waited for
  // inside its branch.  Chunks stay in the state type until they are used.
  constexpr int kPer = kNormChunksPerBlock / kNormThreads;
  constexpr int kBatch = 8;
  static_assert(kPer % kBatch == 0, "batches");
  using R = Raw8<T>;
  float sum = 0.f;
#pragma unroll 1
  for (int i0 = 0; i0 < kPer; i0 += kBatch) {
    typename R::type x[kBatch], y[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int64_t c = c0 + (int64_t)(i0 + i) * kNormThreads + tid;
      x[i] = R::load(src + (c < chunks ? c : chunks - 1) * 8);
    }
    if (ref != nullptr) {
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int64_t c = c0 + (int64_t)(i0 + i) * kNormThreads + tid;
        y[i] = R::load(ref + (c < chunks ? c : chunks - 1) * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const bool ok = c0 + (int64_t)(i0 + i) * kNormThreads + tid < chunks;
      f32x8 v = R::f32(x[i]);
      if (ref != nullptr) v -= R::f32(y[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = ok ? v[e] : 0.f;
        sum = __builtin_fmaf(d, d, sum);
      }
    }
  }
  red[tid] = sum;
  __syncthreads();
#pragma unroll
  for (int off = kNormThreads / 2; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  if (tid == 0) a.partial[(int64_t)si * a.blocks + blockIdx.x] = red[0];
}

__global__ __launch_bounds__(kNormThreads) void norms_final_kernel(const NormArgs a) {
  __shared__ float red[kNormThreads];
  const int tid = threadIdx.x;
  for (int si = 0; si < a.n; ++si) {
    float sum = 0.f;
    for (int b = tid; b < a.blocks; b += kNormThreads) sum += a.partial[(int64_t)si * a.blocks + b];
    red[tid] = sum;
    __syncthreads();
#pragma unroll
    for (int off = kNormThreads / 2; off > 0; off >>= 1) {
      if (tid < off) red[tid] += red[tid + off];
      __syncthreads();
    }
    if (tid == 0) a.norms[si] = __builtin_sqrtf(red[0]);
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_norms(const NormArgs& a, ditango_dtype dt, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.blocks > 0) {
    const dim3 grid((unsigned)a.blocks, (unsigned)a.n);
    if (dt == DITANGO_BF16)
      hipLaunchKernelGGL(norms_partial_kernel<__bf16>, grid, dim3(kNormThreads), 0, s, a);
    else
      hipLaunchKernelGGL(norms_partial_kernel<float>, grid, dim3(kNormThreads), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(norms_final_kernel, dim3(1), dim3(kNormThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ditango

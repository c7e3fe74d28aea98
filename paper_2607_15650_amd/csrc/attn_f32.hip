// attn_f32.hip - fresh attention states of selected key/value partitions,
// float32 inputs and states, float32 MFMA (v_mfma_f32_32x32x2_f32) on gfx950.
//
// Same computation and work decomposition as the bf16 kernel (the blocked
// attention state of Sec. 2.2.4, Eq. attention_state, by online softmax over
// key tiles staged through LDS), in full float32.  Scores are computed
// transposed, S^T = K Q^T, so that each lane holds one query's scores; the
// output is accumulated as O^T = V^T P^T with the probabilities used in
// float32 straight from the score registers.  With one k element per lane
// group per MFMA, V needs no transposition: lane group g of k-step r reads
// the key its score register r holds.
#include "internal.h"

namespace ditango {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32f(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

template <int D, int NW, int BN>
struct CfgF {
  static constexpr int NT = NW * 64;
  static constexpr int BM = NW * 32;          // one 32-row query block per wave
  static constexpr int KS = D / 2;            // MFMA k-steps over the head dim
  static constexpr int KB = BN / 32;
  static constexpr int DB = D / 32;
  static constexpr int KST = D + 1;           // odd stride: conflict-free column reads
  static constexpr int VST = D + 8;
  static constexpr int KTILE = BN * KST;
  static constexpr int VTILE = BN * VST;
  static constexpr int CH = BN * D / 4;       // 16-byte chunks per tile
  static constexpr int CH_T = CH / NT;
  static_assert(CH % NT == 0, "tile not divisible by threads");
};

template <int D, int NW, int BN>
__global__ __launch_bounds__(NW * 64) void attn_f32_kernel(const AttnArgs a) {
  using C = CfgF<D, NW, BN>;
  __shared__ __attribute__((aligned(16))) float smem[2 * (C::KTILE + C::VTILE)];

  const int task = xcd_remap(blockIdx.x, gridDim.x);
  const int qt = task % a.q_tiles;
  int t = task / a.q_tiles;
  const int h = t % a.H;
  t /= a.H;
  const int b = t % a.B;
  const int sel = t / a.B;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 31;
  const int g = lane >> 5;

  const int64_t HD = (int64_t)a.H * D;
  const int kv_len = a.kv_len[sel];
  const int64_t kv0 = a.kv_begin[sel];
  const int slot = a.slot[sel];

  const float* __restrict__ qg = (const float*)a.q;
  const float* __restrict__ kg = (const float*)a.k + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;
  const float* __restrict__ vg = (const float*)a.v + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;

  const int64_t row = (int64_t)qt * C::BM + wave * 32 + lr;
  float qf[C::KS];
  if (row < a.q_len) {
    const float* src = qg + ((int64_t)b * a.q_len + row) * HD + (int64_t)h * D + g;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qf[s] = src[2 * s];
  } else {
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qf[s] = 0.f;
  }

  f32x16 o[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db) o[db] = f32x16{};
  float m = -INFINITY, l = 0.f;

  f32x4 kreg[C::CH_T], vreg[C::CH_T];
  auto load_tile = [&](int key0) {
#pragma unroll
    for (int i = 0; i < C::CH_T; ++i) {
      const int c = tid + i * C::NT;
      const int key = c / (D / 4);
      const int d0 = (c % (D / 4)) * 4;
      if (key0 + key < kv_len) {
        kreg[i] = *(const f32x4*)(kg + (int64_t)(key0 + key) * HD + d0);
        vreg[i] = *(const f32x4*)(vg + (int64_t)(key0 + key) * HD + d0);
      } else {
        kreg[i] = f32x4{};
        vreg[i] = f32x4{};
      }
    }
  };
  auto store_tile = [&](int buf) {
    float* ks = smem + buf * (C::KTILE + C::VTILE);
    float* vs = ks + C::KTILE;
#pragma unroll
    for (int i = 0; i < C::CH_T; ++i) {
      const int c = tid + i * C::NT;
      const int key = c / (D / 4);
      const int d0 = (c % (D / 4)) * 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) ks[key * C::KST + d0 + e] = kreg[i][e];
      *(f32x4*)(vs + key * C::VST + d0) = vreg[i];
    }
  };

  const int n_tiles = (kv_len + BN - 1) / BN;
  if (n_tiles > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  const float sl2 = a.scale_log2;

  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int key0 = it * BN;
    if (it + 1 < n_tiles) load_tile(key0 + BN);
    const float* ks = smem + buf * (C::KTILE + C::VTILE);
    const float* vs = ks + C::KTILE;

    f32x16 sacc[C::KB];
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int s = 0; s < C::KS; ++s)
        sacc[kb] = mfma32f(ks[(kb * 32 + lr) * C::KST + 2 * s + g], qf[s], sacc[kb]);
    }
    if (key0 + BN > kv_len) {
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          if (key >= kv_len) sacc[kb][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx * sl2);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    float ls = 0.f;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][r], sl2, -mnew));
        sacc[kb][r] = p;
        ls += p;
      }
    l = l * alpha + ls;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) o[db] *= alpha;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
          o[db] = mfma32f(vs[key * C::VST + db * 32 + lr], sacc[kb][r], o[db]);
      }

    if (it + 1 < n_tiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  const float lt = l + __shfl_xor(l, 32);
  if (row < a.q_len) {
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    float* outg = (float*)a.out_states;
    const int64_t slot_elems = (int64_t)a.B * a.q_len * HD;
    float* dst = outg + (int64_t)slot * slot_elems + ((int64_t)b * a.q_len + row) * HD +
                 (int64_t)h * D + 4 * g;
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = o[db][4 * r4 + e] * inv;
        *(f32x4*)(dst + db * 32 + 8 * r4) = x;
      }
    if (g == 0) {
      const float lse = lt > 0.f ? (m + __builtin_amdgcn_logf(lt)) * kLn2 : -INFINITY;
      a.lse_states[(((int64_t)slot * a.B + b) * a.H + h) * a.q_len + row] = lse;
    }
  }
}

template <int D, int NW, int BN>
hipError_t launch_cfg_f(const AttnArgs& a0, hipStream_t s) {
  using C = CfgF<D, NW, BN>;
  AttnArgs a = a0;
  a.q_tiles = (int)((a.q_len + C::BM - 1) / C::BM);
  const int64_t nblk = (int64_t)a.q_tiles * a.H * a.B * a.n_sel;
  if (nblk <= 0) return hipSuccess;
  if (nblk > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((attn_f32_kernel<D, NW, BN>), dim3((unsigned)nblk), dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnArgs& a, int D, hipStream_t s) {
  if (D == 128) return launch_cfg_f<128, 4, 32>(a, s);
  if (D == 64) return launch_cfg_f<64, 4, 32>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace ditango

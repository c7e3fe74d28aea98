// attn_bf16.hip - fresh attention states of selected key/value partitions,
// bf16 inputs, bf16 MFMA with float32 accumulation (gfx950).
//
// Computes, for every selected partition j and every query row, the blocked
// attention state of the paper's Sec. 2.2.4 (Eq. attention_state): the
// normalised output OUT_j and LSE_j = log sum exp(scale q.k) over the keys of
// partition j, by a single pass over the keys with a running maximum (online
// softmax).
//
// Work decomposition
//   One workgroup = NW waves = one tile of NW*QB*32 query rows of one
//   (batch, head, selected partition).  Each wave owns QB blocks of 32 query
//   rows.  The workgroup walks the partition's keys in tiles of BN keys; K and
//   V tiles are staged through LDS (double buffered: the global loads of tile
//   i+1 are in flight while tile i is computed) and shared by all waves.
//
// Orientation
//   Scores are computed transposed, S^T = K Q^T, with the 32x32x16 bf16 MFMA:
//   A = K (32 keys x 16 dims, read from LDS), B = Q^T (16 dims x 32 queries,
//   held in registers for the whole kernel).  In the 32x32 accumulator layout
//   each lane then holds 16 keys of a single query (lane % 32), so the row
//   max and row sum are in-register reductions plus one exchange between
//   lanes l and l+32.  The output is likewise accumulated transposed,
//   O^T = V^T P^T: A = V^T (32 dims x 16 keys, from LDS), B = P^T taken
//   straight from the score registers after exp and conversion to bf16.
//   V is stored transposed in LDS, with keys permuted inside each group of 16
//   so that every lane's 8 B-operand keys are one contiguous 16-byte read.
//
// Accumulator layout of the 32x32 MFMA (lane l, register r):
//   row i = 8*(r/4) + 4*(l/32) + (r%4), column j = l % 32.
#include "internal.h"

namespace ditango {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Position of key k (0..15 inside a group of 16) in the transposed V tile:
// 4-key blocks are stored in the order 0,2,1,3 so that lane group g of the
// PV MFMA, which needs keys {4g..4g+3, 8+4g..8+4g+3}, reads 8 contiguous keys.
__device__ __forceinline__ int vperm(int key) {
  const int blk = (key >> 2) & 3;
  const int pblk = ((blk & 1) << 1) | (blk >> 1);
  return (key & ~15) | (pblk << 2) | (key & 3);
}

template <int D, int QB, int NW, int BN>
struct Cfg {
  static constexpr int NT = NW * 64;          // threads per workgroup
  static constexpr int BM = NW * QB * 32;     // query rows per workgroup
  static constexpr int KS = D / 16;           // MFMA k-steps over the head dim
  static constexpr int KB = BN / 32;          // 32-key blocks per key tile
  static constexpr int DB = D / 32;           // 32-dim blocks of the output
  static constexpr int PS = BN / 16;          // MFMA k-steps over a key tile
  static constexpr int KST = D + 8;           // K tile row stride (elements)
  static constexpr int VST = BN + 8;          // V^T tile row stride (elements)
  static constexpr int KTILE = BN * KST;      // elements
  static constexpr int VTILE = D * VST;
  static constexpr int KCH = BN * D / 8;      // 16-byte chunks of a K tile
  static constexpr int KCH_T = KCH / NT;      // per thread
  static constexpr int VPAIRS = (BN / 2) * (D / 8);   // (key pair, 8 dims) items
  static constexpr int VP_T = VPAIRS / NT;
  static_assert(KCH % NT == 0 && VPAIRS % NT == 0, "tile not divisible by threads");
  static_assert(BN % 32 == 0 && D % 32 == 0, "bad tile");
};

template <int D, int QB, int NW, int BN>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(const AttnArgs a) {
  using C = Cfg<D, QB, NW, BN>;
  __shared__ __attribute__((aligned(16))) __bf16 smem[2 * (C::KTILE + C::VTILE)];

  // ---- task decode: (selected partition, batch, head, query tile)
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

  const __bf16* __restrict__ qg = (const __bf16*)a.q;
  const __bf16* __restrict__ kg = (const __bf16*)a.k + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;
  const __bf16* __restrict__ vg = (const __bf16*)a.v + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;

  // ---- Q^T fragments (B operand): lane holds Q[row][16s + 8g .. +8]
  const int64_t row0 = (int64_t)qt * C::BM + wave * (QB * 32);
  bf16x8 qf[QB][C::KS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int64_t row = row0 + qb * 32 + lr;
    if (row < a.q_len) {
      const __bf16* src = qg + ((int64_t)b * a.q_len + row) * HD + (int64_t)h * D + 8 * g;
#pragma unroll
      for (int s = 0; s < C::KS; ++s) qf[qb][s] = *(const bf16x8*)(src + 16 * s);
    } else {
#pragma unroll
      for (int s = 0; s < C::KS; ++s) qf[qb][s] = bf16x8{};
    }
  }

  f32x16 o[QB][C::DB];
  float m[QB], l[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) o[qb][db] = f32x16{};
  }

  // ---- staging registers for one K/V tile
  u32x4 kreg[C::KCH_T];
  u32x4 vreg[C::VP_T][2];

  auto load_tile = [&](int key0) {
#pragma unroll
    for (int i = 0; i < C::KCH_T; ++i) {
      const int c = tid + i * C::NT;
      const int key = c / (D / 8);
      const int d0 = (c % (D / 8)) * 8;
      if (key0 + key < kv_len)
        kreg[i] = *(const u32x4*)(kg + (int64_t)(key0 + key) * HD + d0);
      else
        kreg[i] = u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < C::VP_T; ++i) {
      const int c = tid + i * C::NT;
      const int kp = c % (BN / 2);
      const int d0 = (c / (BN / 2)) * 8;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = key0 + 2 * kp + e;
        if (key < kv_len)
          vreg[i][e] = *(const u32x4*)(vg + (int64_t)key * HD + d0);
        else
          vreg[i][e] = u32x4{0, 0, 0, 0};
      }
    }
  };

  auto store_tile = [&](int buf) {
    __bf16* ks = smem + buf * (C::KTILE + C::VTILE);
    __bf16* vs = ks + C::KTILE;
#pragma unroll
    for (int i = 0; i < C::KCH_T; ++i) {
      const int c = tid + i * C::NT;
      const int key = c / (D / 8);
      const int d0 = (c % (D / 8)) * 8;
      *(u32x4*)(ks + key * C::KST + d0) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < C::VP_T; ++i) {
      const int c = tid + i * C::NT;
      const int kp = c % (BN / 2);
      const int d0 = (c / (BN / 2)) * 8;
      const int pos = vperm(2 * kp);   // keys 2kp, 2kp+1 stay adjacent
      uint32_t* dst = (uint32_t*)(vs + d0 * C::VST + pos);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t x0 = vreg[i][0][w];   // dims d0+2w, d0+2w+1 of key 2kp
        const uint32_t x1 = vreg[i][1][w];   // same dims of key 2kp+1
        // dim d0+2w: (key 2kp, key 2kp+1) low halves; dim d0+2w+1: high halves
        dst[(2 * w) * (C::VST / 2)] = (x0 & 0xffffu) | (x1 << 16);
        dst[(2 * w + 1) * (C::VST / 2)] = (x0 >> 16) | (x1 & 0xffff0000u);
      }
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

    const __bf16* ks = smem + buf * (C::KTILE + C::VTILE);
    const __bf16* vs = ks + C::KTILE;

    // ---- S^T = K Q^T for the tile: sacc[kb][qb] covers keys kb*32..+32
    f32x16 sacc[C::KB][QB];
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sacc[kb][qb] = f32x16{};
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        const bf16x8 ka = *(const bf16x8*)(ks + (kb * 32 + lr) * C::KST + 16 * s + 8 * g);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) sacc[kb][qb] = mfma32(ka, qf[qb][s], sacc[kb][qb]);
      }
    }

    // ---- mask keys past the end of the partition (last tile only)
    if (key0 + BN > kv_len) {
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          if (key >= kv_len) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sacc[kb][qb][r] = -INFINITY;
          }
        }
    }

    // ---- online softmax (base 2, scaled) and P^T fragments
    bf16x8 pf[QB][C::PS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][qb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m[qb], mx * sl2);
      const float alpha = fast_exp2(m[qb] - mnew);
      m[qb] = mnew;
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(__builtin_fmaf(sacc[kb][qb][r], sl2, -mnew));
          sacc[kb][qb][r] = p;
          ls += p;
        }
      l[qb] = l[qb] * alpha + ls;
#pragma unroll
      for (int db = 0; db < C::DB; ++db) o[qb][db] *= alpha;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          f32x8 x;
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = sacc[kb][qb][8 * hh + e];
          pf[qb][2 * kb + hh] = __builtin_convertvector(x, bf16x8);
        }
    }

    // ---- O^T += V^T P^T
#pragma unroll
    for (int s = 0; s < C::PS; ++s) {
#pragma unroll
      for (int db = 0; db < C::DB; ++db) {
        const bf16x8 va = *(const bf16x8*)(vs + (db * 32 + lr) * C::VST + 16 * s + 8 * g);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma32(va, pf[qb][s], o[qb][db]);
      }
    }

    if (it + 1 < n_tiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: normalise, write OUT_j and LSE_j of slot j
  __bf16* outg = (__bf16*)a.out_states;
  const int64_t slot_elems = (int64_t)a.B * a.q_len * HD;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = l[qb] + __shfl_xor(l[qb], 32);
    const int64_t row = row0 + qb * 32 + lr;
    if (row < a.q_len) {
      const float inv = lt > 0.f ? 1.0f / lt : 0.f;
      __bf16* dst = outg + (int64_t)slot * slot_elems + ((int64_t)b * a.q_len + row) * HD +
                    (int64_t)h * D + 4 * g;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 x;
#pragma unroll
          for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
          *(bf16x4*)(dst + db * 32 + 8 * r4) = __builtin_convertvector(x, bf16x4);
        }
      if (g == 0) {
        const float lse = lt > 0.f ? (m[qb] + __builtin_amdgcn_logf(lt)) * kLn2 : -INFINITY;
        a.lse_states[(((int64_t)slot * a.B + b) * a.H + h) * a.q_len + row] = lse;
      }
    }
  }
}

template <int D, int QB, int NW, int BN>
hipError_t launch_cfg(const AttnArgs& a0, hipStream_t s) {
  using C = Cfg<D, QB, NW, BN>;
  AttnArgs a = a0;
  a.q_tiles = (int)((a.q_len + C::BM - 1) / C::BM);
  const int64_t nblk = (int64_t)a.q_tiles * a.H * a.B * a.n_sel;
  if (nblk <= 0) return hipSuccess;
  if (nblk > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((attn_bf16_kernel<D, QB, NW, BN>), dim3((unsigned)nblk), dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int D, hipStream_t s) {
  if (D == 128) return launch_cfg<128, 2, 4, 64>(a, s);
  if (D == 64) return launch_cfg<64, 2, 4, 64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace ditango

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
//   (batch, head, selected partition); a single launch covers every selected
//   partition.  Each wave owns QB blocks of 32 query rows.  The workgroup walks
//   the partition's keys in tiles of BN keys.  K and V tiles go straight from
//   global memory into LDS with the 16-byte direct loads (no staging
//   registers, no LDS write instructions), double buffered, and are shared by
//   all waves of the workgroup.
//
// Orientation
//   Scores are computed transposed, S^T = K Q^T, with the 32x32x16 bf16 MFMA:
//   A = K (32 keys x 16 dims, one 16-byte LDS read per lane), B = Q^T (16 dims
//   x 32 queries, held in registers for the whole kernel).  In the 32x32
//   accumulator layout each lane then holds 16 keys of a single query
//   (lane % 32), so the row max and row sum are in-register reductions plus
//   one exchange between lanes l and l^32.  The output is accumulated
//   transposed too, O^T = V^T P^T: B = P^T comes straight from the score
//   registers after exp2 and conversion to bf16; A = V^T is read from the
//   row-major V tile with the LDS transpose read (ds_read_b64_tr_b16).
//
// LDS layout
//   A K or V tile row (one key, D bf16) is D*2 bytes of 16-byte units; unit c
//   of row `key` is stored at unit c ^ f(key).  The swizzles make the 16-byte
//   K reads (16 consecutive keys, one unit) and the transpose reads of V
//   (4 consecutive keys x 4 units) hit 16 distinct 16-byte bank groups.
//
// Two kernels
//   Launches at D=128, and at D=64 when they run at least four rounds of
//   tasks, use attn_bf16_asm_kernel: four waves, one per SIMD, two 32-row
//   query blocks per wave so that every LDS fragment feeds two MFMAs, the
//   O^T accumulators and Q^T in AGPRs, and a key loop written as gfx950
//   assembly by gen_attn_loop.py (attn_d128_loop.inc, attn_d64_loop.inc).
//   Its fast loop keeps tile 0's maximum for the whole task (no per-tile
//   test); a workgroup whose row sums end above 2^40 or NaN runs its task
//   again in the checked loop, which follows the running-maximum rule below
//   and agrees with the fast loop bit for bit wherever the fast one is kept.
//   The compiled kernel attn_bf16_kernel (the pipeline below) runs the
//   other launches: short D=64 launches, and partitions whose bytes for one
//   head reach the tile loads' 32-bit bounds.
//
// Pipeline of the compiled kernel
//   D=128 (two waves per SIMD): iteration i computes the scores of tile i+1
//   (MFMA) in the same basic block as the exponentials of tile i (VALU), then
//   accumulates P_i V_i (MFMA).  The loads of K_{i+2} and V_{i+1} are in
//   flight during the whole iteration.  D=64 (three waves per SIMD): tile by
//   tile, scores, exponentials and P V of tile i while tile i+1 loads; the
//   other waves of the SIMD overlap the phases.
//
// Running maximum
//   No per-tile row maximum is taken.  Probabilities are computed against the
//   running maximum m as it stands; only a tile whose probabilities grow past
//   2^40 (scores more than 40 above m, base 2, or the first tile, where m is
//   still -inf) is redone after raising m to the tile's row maximum and
//   rescaling the accumulators.  Floating point keeps the relative precision
//   of the large probabilities, and the final normalisation divides the same
//   factor out of OUT and the row sum, so the result does not depend on how
//   far m lags the true maximum.
//
// Accumulator layout of the 32x32 MFMA (lane l, register r):
//   row i = 8*(r/4) + 4*(l/32) + (r%4), column j = l % 32.
#include <type_traits>

#include "internal.h"



namespace ditango {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))
#define GLOBAL_PTR(T, p) ((const __attribute__((address_space(1))) T*)(p))

constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS byte address of a pointer into the workgroup's shared memory
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16-byte direct load global -> LDS for the wave: lane l's 16 bytes from
// base + voff land at LDS byte lds_base + 16*l.  `base` and `lds_base` are
// wave-uniform (scalar registers), `voff` is the lane's byte offset.  Issued
// from inline assembly so that the compiler does not order every later LDS
// read of this wave after it (it cannot tell the DMA target apart from the
// tiles being read); completion is awaited explicitly with s_waitcnt vmcnt
// before the workgroup barrier that publishes the tile.
__device__ __forceinline__ void lds_dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  const uint64_t sbase = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(m0v)
               : "memory", "m0");
}

// max / sum of x over lanes l and l^32 (the two lanes holding one query row)
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1, unrolled
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

template <int D, int QB, int NW, int BN, int NBUF>
struct Cfg {
  static constexpr int NT = NW * 64;          // threads per workgroup
  static constexpr int BM = NW * QB * 32;     // query rows per workgroup
  static constexpr int KS = D / 16;           // MFMA k-steps over the head dim
  static constexpr int KB = BN / 32;          // 32-key blocks per key tile
  static constexpr int DB = D / 32;           // 32-dim blocks of the output
  static constexpr int PS = BN / 16;          // MFMA k-steps over a key tile
  static constexpr int UNITS = D / 8;         // 16-byte units per tile row
  static constexpr int ROWB = D * 2;          // bytes per tile row
  static constexpr int TILEB = BN * ROWB;     // bytes per K or V tile
  static constexpr int LOADS = TILEB / 1024;  // 1 KiB direct loads per tile
  static constexpr int LOADS_W = LOADS / NW;  // per wave
  static constexpr int ROWS_PER_LOAD = 1024 / ROWB;
  static constexpr int PF = NBUF - 1;         // tiles loaded ahead of use
  // vmcnt(n): tile loads a wave may leave in flight at the end of an
  // iteration (those issued in the last PF-1 iterations)
  static constexpr int VM_LEFT = (PF - 1) * 2 * LOADS_W;
  // dynamic LDS: the K and V rings, one Q/OUT staging region per wave and
  // the claimed unit of a queue workgroup
  static constexpr size_t LDS_BYTES = (size_t)2 * NBUF * TILEB + (size_t)NW * QB * 32 * ROWB + 16;
  static_assert(LDS_BYTES <= 163840, "LDS of one compute unit");
  static_assert(NBUF >= 2 && NBUF <= 4, "ring size");   // the unrolled loop keeps slots constant
  static_assert(VM_LEFT <= 63, "vmcnt range");
  static_assert(D == 64 || D == 128, "head dim");
  static_assert(LOADS % NW == 0, "tile loads must split evenly over waves");
  static_assert(BN % 32 == 0, "key tile");
};

// unit swizzles (see the file comment): 16 consecutive keys reading the same
// unit, and 4 consecutive keys x 4 consecutive units, are bank-group distinct
template <int D> __device__ __forceinline__ int swz_k(int key) {
  return D == 128 ? (key & 15) : ((key >> 1) & 7);
}
template <int D> __device__ __forceinline__ int swz_v(int key) {
  return D == 128 ? ((key & 3) << 2) : (((key >> 1) & 1) << 2);
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (expcnt and lgkmcnt not waited for)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// four consecutive output elements of a state row, in the state type
__device__ __forceinline__ void store4(__bf16* p, const f32x4& x) {
  *(bf16x4*)p = __builtin_convertvector(x, bf16x4);
}
__device__ __forceinline__ void store4(float* p, const f32x4& x) { *(f32x4*)p = x; }

// Work units of a launch: the main tasks [0, n_main), then the split units
// n_main + u, u in [0, n_split * split_f) (split task n_main + u / split_f,
// key range u % split_f).  XCD list x holds the x-th contiguous eighth of
// the main tasks, then the x-th eighth of the split units; its first
// n_static / 8 positions run static (workgroup b: position b / 8 of list
// b % 8).  The rest of list x is claimed through two counters: queue x for
// its main tasks, queue 8 + x for its split units.
__device__ __forceinline__ int list_unit(const AttnArgs& a, int x, int t) {
  const int lm = xcd_len(x, a.n_main);
  return t < lm ? xcd_first(x, a.n_main) + t : a.n_main + xcd_first(x, a.n_split * a.split_f) + (t - lm);
}
// first list position and length handed out by queue q (0..15)
__device__ __forceinline__ void queue_range(const AttnArgs& a, int q, int* first, int* len) {
  const int x = q & 7;
  const int s = a.n_static >> 3;
  const int lm = xcd_len(x, a.n_main);
  if (q < 8) {
    *first = min(s, lm);
    *len = lm - *first;
  } else {
    *first = max(s, lm);
    *len = lm + xcd_len(x, a.n_split * a.split_f) - *first;
  }
}

// Claims one unit for a workgroup past the static ones (called by all 64
// lanes of its first wave; the result is wave-uniform).  Main tasks go
// before split units, so that no short unit runs while a full task waits:
// this XCD's main queue; then, from one look at all the counters, the main
// queue with the most left; then this XCD's split queue, then the split
// queue with the most left; finally every queue in turn.  Counters only
// grow, so a queue seen exhausted stays so, and -1 (nothing left) is
// returned only after every queue was seen exhausted.
__device__ int claim_unit(const AttnArgs& a, int lane) {
  unsigned xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  const int own = (int)(xcc & 7);
  // one atomic increment of queue q (wave-uniform) by lane 0
  auto take = [&](int q) -> int {
    int first, len;
    queue_range(a, q, &first, &len);
    if (len <= 0) return -1;
    int t = 0;
    if (lane == 0) t = __hip_atomic_fetch_add(a.queue + q, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    t = __builtin_amdgcn_readfirstlane(t);
    return t < len ? list_unit(a, q & 7, first + t) : -1;
  };
  int u = take(own);
  if (u >= 0) return u;
  bool own_split_tried = false;
  for (int it = 0; it < 4; ++it) {
    int left = 0;
    if (lane < 16) {
      int first, len;
      queue_range(a, lane, &first, &len);
      left = len - __hip_atomic_load(a.queue + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // the queue with the most left among lanes 0..7 (main), else among
    // lanes 8..15 (split): max of (left, lane) within each group of 8
    int key = left > 0 ? (left << 4) | lane : -1;
    key = max(key, __shfl_xor(key, 1));
    key = max(key, __shfl_xor(key, 2));
    key = max(key, __shfl_xor(key, 4));
    const int main_key = __builtin_amdgcn_readlane(key, 0);
    const int split_key = __builtin_amdgcn_readlane(key, 8);
    int q;
    if (main_key >= 0) {
      q = main_key & 15;
    } else if (!own_split_tried && __builtin_amdgcn_readlane(left, 8 + own) > 0) {
      q = 8 + own;
      own_split_tried = true;
    } else if (split_key >= 0) {
      q = split_key & 15;
    } else {
      return -1;
    }
    u = take(q);
    if (u >= 0) return u;
  }
  for (int k = 1; k < 16; ++k) {
    u = take(k < 8 ? (own + k) & 7 : 8 + ((own + k) & 7));
    if (u >= 0) return u;
  }
  return -1;
}

template <int D, int QB, int NW, int BN, int NBUF, int WPE, bool SEQ, typename TS>
__global__ __launch_bounds__(NW * 64, WPE) void attn_bf16_kernel(const AttnArgs a) {
  using C = Cfg<D, QB, NW, BN, NBUF>;
  // LDS: the K and V rings (2*NBUF tiles), then one staging region per wave
  // (its QB*32 rows of Q on the way in, of OUT on the way out), then one
  // int: the claimed unit of a queue workgroup
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  constexpr int kStage = 2 * NBUF * C::TILEB;
  constexpr int kStageWave = QB * 32 * C::ROWB;

  // ---- task decode: (selected partition, batch, head, query tile), and for
  // a task of the split tail, which of its split_f key ranges
  int u;
  if ((int)blockIdx.x < a.n_static) {
    u = list_unit(a, (int)blockIdx.x & 7, (int)blockIdx.x >> 3);
  } else {
    int* claimed = (int*)(smem + kStage + NW * kStageWave);
    if (threadIdx.x < 64) {
      const int c = claim_unit(a, (int)threadIdx.x);
      if (threadIdx.x == 0) *claimed = c;
    }
    __syncthreads();
    u = __builtin_amdgcn_readfirstlane(*claimed);
    if (u < 0) return;
  }
  int task = u, part = -1;
  if (u >= a.n_main) {
    task = a.n_main + (u - a.n_main) / a.split_f;
    part = (u - a.n_main) % a.split_f;
  }
  const int qt = task % a.q_tiles;
  int t = task / a.q_tiles;
  const int h = t % a.H;
  t /= a.H;
  const int b = t % a.B;
  const int sel = t / a.B;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar registers
  const int lr = lane & 31;
  const int g = lane >> 5;

  const int64_t HD = (int64_t)a.H * D;
  int kv_len = a.kv_len[sel];
  int64_t kv0 = a.kv_begin[sel];
  const int slot = a.slot[sel];
  if (part >= 0) {
    // key range `part` of split_f: whole tiles, the last range the remainder
    const int per = ((kv_len + BN - 1) / BN + a.split_f - 1) / a.split_f * BN;
    const int k0 = min(part * per, kv_len);
    const int k1 = min(k0 + per, kv_len);
    kv0 += k0;
    kv_len = k1 - k0;
  }

  const __bf16* __restrict__ qg = (const __bf16*)a.q;
  const __bf16* __restrict__ kg = (const __bf16*)a.k + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;
  const __bf16* __restrict__ vg = (const __bf16*)a.v + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;

  // ---- Q^T fragments (B operand): lane holds Q[row][16s + 8g .. +8].  The
  // wave's QB*32 query rows come in through its LDS staging region, loaded
  // like a K tile (whole rows per 1 KiB load, units swizzled by row), and are
  // read back once the loads have landed (unstage_q).
  const int64_t row0 = (int64_t)qt * C::BM + wave * (QB * 32);
  bf16x8 qf[QB][C::KS];
  const unsigned char* stage = smem + kStage + wave * kStageWave;
  // 16-byte unit swizzle of an OUT row staged for the store: rows r..r+15
  // of one accumulator register land in distinct bank groups (rows r and
  // r + 16 also swap the two 8-byte halves of a unit)
  auto swz_out = [](int row) { return row & (C::UNITS - 1); };
  auto unstage_q = [&]() {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int s = 0; s < C::KS; ++s)
        qf[qb][s] = *(const bf16x8*)(stage + (qb * 32 + lr) * C::ROWB +
                                     (((2 * s + g) ^ swz_k<D>(qb * 32 + lr)) * 16));
  };

  f32x16 o[QB][C::DB];
  float m[QB], l[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) o[qb][db] = f32x16{};
  }

  // ---- direct global -> LDS tile loads.  Lane l of a 1 KiB load writes LDS
  // unit l of that KiB, i.e. row l / UNITS, stored unit l % UNITS; it fetches
  // the global unit that the swizzle maps there.  The lane's byte offset from
  // the tile's first key is the same for every tile, so it is computed once;
  // the tile base is wave-uniform.  Rows past the end of the partition are
  // clamped to its last key: their scores are masked to -inf and their
  // probabilities are exactly 0, so any finite value will do, and every load
  // stays inside the partition.
  const int last_key = kv_len > 0 ? kv_len - 1 : 0;
  const int ld_row = lane / C::UNITS;
  const int ld_unit = lane % C::UNITS;
  const uint32_t row_bytes = (uint32_t)HD * 2;
  uint32_t ld_off_k[C::LOADS_W], ld_off_v[C::LOADS_W];
#pragma unroll
  for (int i = 0; i < C::LOADS_W; ++i) {
    const int row = (wave * C::LOADS_W + i) * C::ROWS_PER_LOAD + ld_row;   // tile row (key)
    ld_off_k[i] = row * row_bytes + (uint32_t)((ld_unit ^ swz_k<D>(row)) * 16);
    ld_off_v[i] = row * row_bytes + (uint32_t)((ld_unit ^ swz_v<D>(row)) * 16);
  }
  const uint32_t smem_lds = lds_addr(smem);
  if (kv_len > 0) {
    // rows past q_len are clamped to the last row: computed, never stored
    const int64_t rb0 = min(row0, a.q_len - 1);
    const __bf16* base = qg + ((int64_t)b * a.q_len + rb0) * HD + (int64_t)h * D;
    const uint32_t dst = smem_lds + (uint32_t)(kStage + wave * kStageWave);
#pragma unroll
    for (int i = 0; i < kStageWave / 1024; ++i) {
      const int row = i * C::ROWS_PER_LOAD + ld_row;
      const int64_t gr = min(row0 + row, a.q_len - 1) - rb0;
      lds_dma16(base, (uint32_t)gr * row_bytes + (uint32_t)((ld_unit ^ swz_k<D>(row)) * 16), dst + (uint32_t)(i * 1024));
    }
  }
  auto load_tile = [&](const __bf16* src, uint32_t dst, int key0, bool is_k) {
    if (key0 + BN <= kv_len) {
      const __bf16* base = src + (int64_t)key0 * HD;
#pragma unroll
      for (int i = 0; i < C::LOADS_W; ++i)
        lds_dma16(base, is_k ? ld_off_k[i] : ld_off_v[i], dst + (wave * C::LOADS_W + i) * 1024);
    } else {
      // the partition's last tile (or one past its end): clamp every row
      const int key_b = min(key0, last_key);
      const __bf16* base = src + (int64_t)key_b * HD;
#pragma unroll
      for (int i = 0; i < C::LOADS_W; ++i) {
        const int li = wave * C::LOADS_W + i;
        const int row = li * C::ROWS_PER_LOAD + ld_row;
        const int key = min(key0 + row, last_key) - key_b;
        const int unit = ld_unit ^ (is_k ? swz_k<D>(row) : swz_v<D>(row));
        lds_dma16(base, (uint32_t)key * row_bytes + (uint32_t)(unit * 16), dst + li * 1024);
      }
    }
  };

  // rings of NBUF K tiles and NBUF V tiles (LDS byte addresses): tile t lives
  // in slot t % NBUF
  auto kbuf_lds = [&](int t) { return smem_lds + (uint32_t)((t % NBUF) * C::TILEB); };
  auto vbuf_lds = [&](int t) { return smem_lds + (uint32_t)((NBUF + t % NBUF) * C::TILEB); };
  auto kbuf = [&](int t) { return smem + (t % NBUF) * C::TILEB; };
  auto vbuf = [&](int t) { return smem + (NBUF + t % NBUF) * C::TILEB; };

  // K A-operand: lane reads unit (2s + g) of row kb*32 + lr
  const int krow_off = lr * C::ROWB;
  const int kswz = swz_k<D>(lr);
  // V^T A-operand by transpose reads: in each 16-lane group, source lane r
  // points at row 4g + r/4 (+ 16s + 8hh) and dims 32db + 16*(group%2) + 4*(r%4);
  // lane i of the group then receives 4 consecutive keys at dim 16*(group%2) + i.
  const int grp = lane >> 4;
  const int rr = lane & 15;
  const int vrow = 4 * g + (rr >> 2);                       // + 16s + 8hh
  const int vdim = 16 * (grp & 1) + 4 * (rr & 3);           // + 32db
  int voff[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db) {
    const int dim = 32 * db + vdim;
    const int unit = (dim >> 3) ^ swz_v<D>(vrow);           // swizzle depends on row % 4 only
    voff[db] = vrow * C::ROWB + unit * 16 + (dim & 7) * 2;
  }

  // S^T = K Q^T of one key tile
  auto qk = [&](const unsigned char* ks, f32x16 (&sacc)[C::KB][QB]) {
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sacc[kb][qb] = f32x16{};
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        const int unit = (2 * s + g) ^ kswz;                 // kb*32 keeps row % 16
        const bf16x8 ka = *(const bf16x8*)(ks + kb * 32 * C::ROWB + krow_off + unit * 16);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) sacc[kb][qb] = mfma32(ka, qf[qb][s], sacc[kb][qb]);
      }
    }
  };
  auto v_frag = [&](const unsigned char* vs, int s, int db) {
    const unsigned char* p = vs + 16 * s * C::ROWB + voff[db];
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, p));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, p + 8 * C::ROWB));
    const u32x2 l2 = __builtin_bit_cast(u32x2, lo);
    const u32x2 h2 = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
  };
  // keys at or past the end of the partition -> -inf
  auto mask_tail = [&](f32x16 (&sacc)[C::KB][QB], int key0) {
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
  };

  const float sl2 = a.scale_log2;
  // Probabilities are taken against a running maximum m that is raised only
  // when a tile's probabilities grow large: exp2(s*scale*log2e - m) for every
  // score of the tile, with this lane's partial row sums in ls.
  auto softmax_tile = [&](const f32x16 (&sc)[C::KB][QB], bf16x8 (&pf)[QB][C::PS], float (&ls)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float sum = 0.f;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          f32x8 x;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            x[e] = fast_exp2(__builtin_fmaf(sc[kb][qb][8 * hh + e], sl2, -m[qb]));
            sum += x[e];
          }
          pf[qb][2 * kb + hh] = __builtin_convertvector(x, bf16x8);
        }
      ls[qb] = sum;
    }
  };
  // A tile whose probabilities against m sum past 2^40 in some lane (its
  // scores exceed m by more than 40, base 2), or hold an inf or a NaN (the
  // first tile: m = -inf), is redone: m is raised to the row maximum of the
  // tile, O and l are rescaled, and the probabilities recomputed.  Otherwise
  // probabilities stay below 2^40 and the row sum below 2^40 times the key
  // count, well inside float32; OUT = O / l and LSE = m + log2 l do not
  // depend on which m was used.  So no tile maximum is taken in the common
  // case.
  constexpr float kBig = 1099511627776.0f;   // 2^40
  auto softmax_checked = [&](const f32x16 (&sc)[C::KB][QB], bf16x8 (&pf)[QB][C::PS]) {
    float ls[QB];
    softmax_tile(sc, pf, ls);
    bool big = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) big |= !(ls[qb] <= kBig);
    if (__builtin_amdgcn_ballot_w64(big) != 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][qb][r]);
        const float mnew = fmaxf(m[qb], pair_max(mx) * sl2);
        const float alpha = m[qb] == -INFINITY ? 0.f : fast_exp2(m[qb] - mnew);
        m[qb] = mnew;
        l[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) o[qb][db] *= alpha;
      }
      softmax_tile(sc, pf, ls);
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l[qb] += ls[qb];
  };

  // O^T += V^T P^T over the key steps of a tile; the V operands of key step
  // s+1 are read while the MFMAs of step s run
  auto pv = [&](const unsigned char* v_cur, const bf16x8 (&pf)[QB][C::PS]) {
    bf16x8 va[2][C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db) va[0][db] = v_frag(v_cur, 0, db);
#pragma unroll
    for (int s = 0; s < C::PS; ++s) {
      if (s + 1 < C::PS) {
#pragma unroll
        for (int db = 0; db < C::DB; ++db) va[(s + 1) & 1][db] = v_frag(v_cur, s + 1, db);
      }
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma32(va[s & 1][db], pf[qb][s], o[qb][db]);
    }
  };

  // One pipelined iteration over key tile i.  On entry S_i holds the scores
  // of tile i.  Block A: the MFMAs of S_{i+1} = K_{i+1} Q^T run while the VALU
  // turns S_i into probabilities P_i (exp2, row sums, bf16).  Block B: the
  // MFMAs of O += V_i P_i.
  // `ph` (a compile-time constant, i % NBUF) fixes every ring slot the
  // iteration touches, so LDS addresses are constant offsets of one base.
  auto iteration = [&](int i, auto ph, f32x16 (&scur)[C::KB][QB], f32x16 (&snxt)[C::KB][QB]) {
    constexpr int P0 = decltype(ph)::value;
    const unsigned char* k_next = smem + ((P0 + 1) % NBUF) * C::TILEB;
    const unsigned char* v_cur = smem + (NBUF + P0) * C::TILEB;
    // Tile i is the partition's last and partial: mask its keys past the end.
    if ((i + 1) * BN > kv_len) mask_tail(scur, i * BN);
    // K_{i+1+PF} and V_{i+PF} land in LDS during the next PF iterations; they
    // overwrite K_{i+1+PF-NBUF} and V_{i+PF-NBUF}, consumed before the last
    // barrier
    load_tile(kg, smem_lds + (uint32_t)(((P0 + 1 + C::PF) % NBUF) * C::TILEB), (i + 1 + C::PF) * BN, true);
    load_tile(vg, smem_lds + (uint32_t)((NBUF + (P0 + C::PF) % NBUF) * C::TILEB), (i + C::PF) * BN, false);
    qk(k_next, snxt);
    bf16x8 pf[QB][C::PS];
    softmax_checked(scur, pf);
    pv(v_cur, pf);
    // K_{i+2} and V_{i+1}, used by the next iteration, have landed for this
    // wave; the barrier makes that true for the whole workgroup
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(C::VM_LEFT));
    __syncthreads();
  };

  const int n_tiles = (kv_len + BN - 1) / BN;
  if constexpr (SEQ) {
    // Tile by tile: scores, probabilities, PV.  Used with three waves per
    // SIMD, where the other waves of the SIMD fill the MFMA and VALU gaps of
    // each wave's dependent sequence and the smaller register footprint of
    // this loop is what allows the third wave.
    if (n_tiles > 0) {
#pragma unroll
      for (int j = 0; j < C::PF; ++j) {
        load_tile(kg, kbuf_lds(j), j * BN, true);
        load_tile(vg, vbuf_lds(j), j * BN, false);
      }
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(C::VM_LEFT));   // the queries and tile 0 have landed
      unstage_q();
      __syncthreads();
      for (int i = 0; i < n_tiles; ++i) {
        // tile i+PF replaces tile i+PF-NBUF, consumed before the last barrier
        load_tile(kg, kbuf_lds(i + C::PF), (i + C::PF) * BN, true);
        load_tile(vg, vbuf_lds(i + C::PF), (i + C::PF) * BN, false);
        f32x16 sc[C::KB][QB];
        qk(kbuf(i), sc);
        if ((i + 1) * BN > kv_len) mask_tail(sc, i * BN);
        bf16x8 pf[QB][C::PS];
        softmax_checked(sc, pf);
        pv(vbuf(i), pf);
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(C::VM_LEFT));   // tile i+1 has landed
        __syncthreads();
      }
    }
  } else {
    f32x16 s0[C::KB][QB], s1[C::KB][QB];
    if (n_tiles > 0) {
      // K_0, then the loads iterations -PF..-1 would have issued, in the same
      // order as the loop issues them
      load_tile(kg, kbuf_lds(0), 0, true);
#pragma unroll
      for (int j = -C::PF; j < 0; ++j) {
        load_tile(kg, kbuf_lds(j + 1 + C::PF), (j + 1 + C::PF) * BN, true);
        load_tile(vg, vbuf_lds(j + C::PF), (j + C::PF) * BN, false);
      }
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(C::VM_LEFT));   // the queries, K_0, K_1, V_0 have landed
      unstage_q();
      __syncthreads();
      qk(kbuf(0), s0);
      // every wave has read K_0 before iteration 0 loads K_2 into its slot
      __syncthreads();
      // K_i is consumed one iteration early (scores of the next tile).  The
      // loop is unrolled over U tiles, a multiple of both the ring size and
      // the two score buffers, so that every ring slot is a constant.
      constexpr int U = NBUF % 2 == 0 ? NBUF : 2 * NBUF;
      for (int i = 0; i < n_tiles; i += U) {
        static_for<U>([&](auto u) {
          constexpr int k = decltype(u)::value;
          if (k == 0 || i + k < n_tiles) {
            if constexpr (k % 2 == 0)
              iteration(i + k, std::integral_constant<int, k % NBUF>{}, s0, s1);
            else
              iteration(i + k, std::integral_constant<int, k % NBUF>{}, s1, s0);
          }
        });
      }
    }
  }

  // ---- epilogue: normalise, write OUT_j and LSE_j of slot j (a split
  // task's range: its partial state, in float32, to the workspace)
  TS* outg = (TS*)a.out_states;
  const int64_t slot_elems = (int64_t)a.B * a.q_len * HD;
  const int64_t pt = part >= 0 ? (int64_t)(task - a.n_main) * a.split_f + part : 0;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = pair_sum(l[qb]);
    const int64_t row = row0 + qb * 32 + lr;
    if (row < a.q_len) {
      const float inv = lt > 0.f ? 1.0f / lt : 0.f;
      const float lse = lt > 0.f ? (m[qb] + __builtin_amdgcn_logf(lt)) * kLn2 : -INFINITY;
      if (part < 0) {
        if constexpr (sizeof(TS) == 2 && D == 128) {
          // bf16 states: into the wave's staging region (row-major, 16-byte
          // units swizzled by row), stored below as whole rows
          unsigned char* srow = (unsigned char*)stage + (qb * 32 + lr) * C::ROWB;
#pragma unroll
          for (int db = 0; db < C::DB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              f32x4 x;
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
              // rows r and r + 16 share a unit, so they take opposite halves
              const int unit = (4 * db + r4) ^ swz_out(qb * 32 + lr);
              const int half = g ^ ((lr >> 4) & 1);
              *(bf16x4*)(srow + unit * 16 + 8 * half) = __builtin_convertvector(x, bf16x4);
            }
        } else {
          TS* dst = outg + (int64_t)slot * slot_elems + ((int64_t)b * a.q_len + row) * HD +
                        (int64_t)h * D + 4 * g;
#pragma unroll
          for (int db = 0; db < C::DB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              f32x4 x;
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
              store4(dst + db * 32 + 8 * r4, x);
            }
        }
        if (g == 0) a.lse_states[(((int64_t)slot * a.B + b) * a.H + h) * a.q_len + row] = lse;
      } else {
        const int64_t rl = row - (int64_t)qt * C::BM;            // row within the query tile
        float* dst = a.part_out + (pt * C::BM + rl) * D + 4 * g;
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            f32x4 x;
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
            store4(dst + db * 32 + 8 * r4, x);
          }
        if (g == 0) a.part_lse[pt * C::BM + rl] = lse;
      }
    }
  }
  if constexpr (sizeof(TS) == 2 && D == 128) {
    if (part < 0) {
      // the staged rows, whole: lane l stores unit l % UNITS of row
      // l / UNITS + ROWS_PER_LOAD * i (the wave's own region, so its LDS
      // writes above are visible to these reads without a barrier)
      TS* dst0 = outg + (int64_t)slot * slot_elems + (int64_t)b * a.q_len * HD + (int64_t)h * D + ld_unit * 8;
#pragma unroll
      for (int i = 0; i < QB * 32 / C::ROWS_PER_LOAD; ++i) {
        const int row = i * C::ROWS_PER_LOAD + ld_row;
        if (row0 + row < a.q_len) {
          bf16x8 x = *(const bf16x8*)(stage + row * C::ROWB + ((ld_unit ^ swz_out(row)) * 16));
          if ((row >> 4) & 1) x = __builtin_shufflevector(x, x, 4, 5, 6, 7, 0, 1, 2, 3);
          *(bf16x8*)(dst0 + (row0 + row) * HD) = x;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The hand-scheduled key loop (attn_d128_loop.inc, attn_d64_loop.inc, written
// by gen_attn_loop.py, whose docstring describes the schedule).  One wave per
// SIMD, two 32-row query blocks per wave: 4 waves, 256 query rows per
// workgroup, 64-key tiles in a 4-deep LDS ring (K first, then V).  Task
// decode, split units and the epilogue are those of attn_bf16_kernel; the
// loop keeps every value in fixed registers, which the asm statement's
// operands pin.
#include "attn_d128_loop.inc"
#include "attn_d64_loop.inc"

template <int D_>
struct AsmCfg {
  static constexpr int D = D_, QB = 2, NW = 4, BN = 64;
  static constexpr int NT = NW * 64;
  static constexpr int BM = NW * QB * 32;     // 256 rows
  static constexpr int KS = D / 16;           // MFMA k-steps over the head dim
  static constexpr int DB = D / 32;           // 32-dim blocks of the output
  static constexpr int ROWB = D * 2;
  static constexpr int UNITS = D / 8;
  static constexpr int ROWS_PER_LOAD = 1024 / ROWB;
  static constexpr int TILEB = BN * ROWB;
  static constexpr int LW = TILEB / 1024 / NW;   // 1 KiB loads per wave per tile
  static constexpr int RING = 8 * TILEB;      // K ring (4 tiles), then V ring (4 tiles)
  static constexpr size_t LDS_BYTES = RING + 16;
  static_assert(QB * 32 * ROWB * NW <= RING, "output staging inside the ring");
};

// Bound on a lane's row sum below which the fast key loop's result is the
// checked loop's, bit for bit (the checked loop raises m only for a tile
// whose sum passes it).
constexpr float kRowSumBound = 1099511627776.0f;   // 2^40

// Buffer descriptor of raw bytes [base, base + nbytes): out-of-range loads
// return zeros and do not access memory.  Word 3 selects 32-bit data format
// for the gfx9 family.
__device__ __forceinline__ u32x4 raw_buffer_desc(const void* base, uint32_t nbytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p),
               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) & 0xffffu,
               (uint32_t)__builtin_amdgcn_readfirstlane(nbytes), 0x00020000u};
}

template <int D_, typename TS>
__global__ __launch_bounds__(256, 1) void attn_bf16_asm_kernel(const AttnArgs a) {
  using C = AsmCfg<D_>;
  constexpr int D = C::D, QB = C::QB, BN = C::BN, KS = C::KS, DB = C::DB, LW = C::LW;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];

  int u;
  if ((int)blockIdx.x < a.n_static) {
    u = list_unit(a, (int)blockIdx.x & 7, (int)blockIdx.x >> 3);
  } else {
    int* claimed = (int*)(smem + C::RING);
    if (threadIdx.x < 64) {
      const int c = claim_unit(a, (int)threadIdx.x);
      if (threadIdx.x == 0) *claimed = c;
    }
    __syncthreads();
    u = __builtin_amdgcn_readfirstlane(*claimed);
    if (u < 0) return;
  }
  int task = u, part = -1;
  if (u >= a.n_main) {
    task = a.n_main + (u - a.n_main) / a.split_f;
    part = (u - a.n_main) % a.split_f;
  }
  const int qt = task % a.q_tiles;
  int t = task / a.q_tiles;
  const int h = t % a.H;
  t /= a.H;
  const int b = t % a.B;
  const int sel = t / a.B;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31;
  const int g = lane >> 5;

  const int64_t HD = (int64_t)a.H * D;
  int kv_len = a.kv_len[sel];
  int64_t kv0 = a.kv_begin[sel];
  const int slot = a.slot[sel];
  if (part >= 0) {
    const int per = ((kv_len + BN - 1) / BN + a.split_f - 1) / a.split_f * BN;
    const int k0 = min(part * per, kv_len);
    const int k1 = min(k0 + per, kv_len);
    kv0 += k0;
    kv_len = k1 - k0;
  }
  const int64_t row0 = (int64_t)qt * C::BM + wave * (QB * 32);
  const uint32_t row_bytes = (uint32_t)HD * 2;

  f32x16 o[QB][DB];
  float m[QB], l[QB];
  if (kv_len > 0) {
    const uint32_t smem_lds = lds_addr(smem);
    // bytes from the partition's first key (this head) to the end of its last
    const uint32_t nrec = (uint32_t)(kv_len - 1) * row_bytes + C::ROWB;
    // this lane's LDS addresses: K fragment of k-step s (row lr, unit
    // (2s+g) ^ swizzle), V^T transpose reads of dim block db
    uint32_t kaddr[KS], vaddr[DB], dmak[LW], dmav[LW];
#pragma unroll
    for (int s = 0; s < KS; ++s) kaddr[s] = smem_lds + lr * C::ROWB + (uint32_t)(((2 * s + g) ^ swz_k<D>(lr)) * 16);
    const int grp = lane >> 4, rr = lane & 15;
    const int vrow = 4 * g + (rr >> 2);
    const int vdim = 16 * (grp & 1) + 4 * (rr & 3);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int dim = 32 * db + vdim;
      vaddr[db] = smem_lds + C::RING / 2 + vrow * C::ROWB + (uint32_t)((((dim >> 3) ^ swz_v<D>(vrow))) * 16) + (dim & 7) * 2;
    }
    // tile loads: lane l of load j writes LDS unit l of the wave's j-th KiB
    // (row l / UNITS of the ROWS_PER_LOAD the KiB holds, stored unit
    // l % UNITS) from the global unit the swizzle maps there.  Load j carries
    // j KiB as its immediate offset, which the hardware adds to the LDS
    // destination and to the global address (and to the offset it range
    // checks), so the lane's register holds its byte offset minus j KiB
    // (never negative: the rows of the j-th KiB start j KiB of key rows in).
    const int ld_row = lane / C::UNITS, ld_unit = lane % C::UNITS;
#pragma unroll
    for (int j = 0; j < LW; ++j) {
      const int row = (wave * LW + j) * C::ROWS_PER_LOAD + ld_row;
      dmak[j] = row * row_bytes + (uint32_t)((ld_unit ^ swz_k<D>(row)) * 16) - 1024u * j;
      dmav[j] = row * row_bytes + (uint32_t)((ld_unit ^ swz_v<D>(row)) * 16) - 1024u * j;
    }
    const float sl2 = a.scale_log2;
    const uint32_t ntiles = (uint32_t)((kv_len + BN - 1) / BN);
    const uint32_t kvl = (uint32_t)kv_len;
    const uint32_t wlds = __builtin_amdgcn_readfirstlane(smem_lds + (uint32_t)wave * (LW * 1024u));
    const uint32_t tileb = __builtin_amdgcn_readfirstlane(row_bytes * BN);
    // Two forms of the key loop.  The fast one takes the running maximum m
    // from tile 0 and keeps it; the checked one tests every tile and raises
    // m (slow path) where a lane's tile sum passes 2^40 or is not a number.
    // Both give m the same value at tile 0, so while no tile of the checked
    // form would take the slow path the two agree bit for bit, and that is
    // the case exactly when every lane's row sum (its tile sums added up)
    // stays within 2^40: the fast form runs first, and a workgroup in which
    // some lane's row sum left that range (or is NaN) runs its task again in
    // the checked form.
    int* redo = (int*)(smem + C::RING) + 1;
    if (tid == 0) *redo = 0;
    for (int pass = 0; pass < 2; ++pass) {
      const __bf16* kp = (const __bf16*)a.k + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;
      const __bf16* vp = (const __bf16*)a.v + ((int64_t)b * a.S + kv0) * HD + (int64_t)h * D;
      u32x4 kd = raw_buffer_desc(kp, nrec);
      u32x4 vd = raw_buffer_desc(vp, nrec);
      // the lane's Q rows (rows past q_len clamped: computed, never stored),
      // advanced to dims 8g..8g+7
      uint64_t qptr0, qptr1;
      {
        const __bf16* qb0 = (const __bf16*)a.q + ((int64_t)b * a.q_len + min(row0 + lr, a.q_len - 1)) * HD + (int64_t)h * D + 8 * g;
        const __bf16* qb1 = (const __bf16*)a.q + ((int64_t)b * a.q_len + min(row0 + 32 + lr, a.q_len - 1)) * HD + (int64_t)h * D + 8 * g;
        qptr0 = (uint64_t)(uintptr_t)qb0;
        qptr1 = (uint64_t)(uintptr_t)qb1;
      }
      if constexpr (D == 128) {
#define DITANGO_D128_CALL(BODY)                                                                                       \
  asm volatile(BODY                                                                                                   \
               : "={a[0:15]}"(o[0][0]), "={a[16:31]}"(o[0][1]), "={a[32:47]}"(o[0][2]), "={a[48:63]}"(o[0][3]),      \
                 "={a[64:79]}"(o[1][0]), "={a[80:95]}"(o[1][1]), "={a[96:111]}"(o[1][2]), "={a[112:127]}"(o[1][3]),   \
                 "={v230}"(m[0]), "={v231}"(m[1]), "={v232}"(l[0]), "={v233}"(l[1]),                                  \
                 "+{s[48:51]}"(kd), "+{s[52:55]}"(vd), "+{v[64:65]}"(qptr0), "+{v[66:67]}"(qptr1)                     \
               : "{v234}"(kaddr[0]), "{v235}"(kaddr[1]), "{v236}"(kaddr[2]), "{v237}"(kaddr[3]),                      \
                 "{v238}"(kaddr[4]), "{v239}"(kaddr[5]), "{v240}"(kaddr[6]), "{v241}"(kaddr[7]),                      \
                 "{v242}"(vaddr[0]), "{v243}"(vaddr[1]), "{v244}"(vaddr[2]), "{v245}"(vaddr[3]),                      \
                 "{v246}"(dmak[0]), "{v247}"(dmak[1]), "{v248}"(dmak[2]), "{v249}"(dmak[3]),                          \
                 "{v250}"(dmav[0]), "{v251}"(dmav[1]), "{v252}"(dmav[2]), "{v253}"(dmav[3]),                          \
                 "{s40}"(sl2), "{s41}"(ntiles), "{s42}"(kvl), "{s44}"(wlds), "{s45}"(tileb)             \
               : DITANGO_D128_LOOP_CLOBBERS)
        if (pass == 0) {
          DITANGO_D128_CALL(DITANGO_D128_FAST_ASM);
        } else {
          DITANGO_D128_CALL(DITANGO_D128_LOOP_ASM);
        }
#undef DITANGO_D128_CALL
      } else {
#define DITANGO_D64_CALL(BODY)                                                                                        \
  asm volatile(BODY                                                                                                   \
               : "={a[0:15]}"(o[0][0]), "={a[16:31]}"(o[0][1]), "={a[32:47]}"(o[1][0]), "={a[48:63]}"(o[1][1]),      \
                 "={v230}"(m[0]), "={v231}"(m[1]), "={v232}"(l[0]), "={v233}"(l[1]),                                  \
                 "+{s[48:51]}"(kd), "+{s[52:55]}"(vd), "+{v[64:65]}"(qptr0), "+{v[66:67]}"(qptr1)                     \
               : "{v234}"(kaddr[0]), "{v235}"(kaddr[1]), "{v236}"(kaddr[2]), "{v237}"(kaddr[3]),                      \
                 "{v238}"(vaddr[0]), "{v239}"(vaddr[1]), "{v240}"(dmak[0]), "{v241}"(dmak[1]),                        \
                 "{v242}"(dmav[0]), "{v243}"(dmav[1]),                                                                \
                 "{s40}"(sl2), "{s41}"(ntiles), "{s42}"(kvl), "{s44}"(wlds), "{s45}"(tileb)             \
               : DITANGO_D64_LOOP_CLOBBERS)
        if (pass == 0) {
          DITANGO_D64_CALL(DITANGO_D64_FAST_ASM);
        } else {
          DITANGO_D64_CALL(DITANGO_D64_LOOP_ASM);
        }
#undef DITANGO_D64_CALL
      }
      // every wave's loads have landed and its reads of the ring are done
      // before the ring is reused (output rows, or the checked pass)
      __syncthreads();
      if (pass == 1) break;
      const bool over = !(l[0] <= kRowSumBound && l[1] <= kRowSumBound);
      if (__builtin_amdgcn_ballot_w64(over) != 0 && lane == 0) *redo = 1;
      __syncthreads();
      if (__builtin_amdgcn_readfirstlane(*redo) == 0) break;
    }
  } else {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      m[qb] = -INFINITY;
      l[qb] = 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[qb][db] = f32x16{};
    }
  }

  // ---- epilogue (as attn_bf16_kernel): the wave's staging region is the
  // start of its K ring slot
  unsigned char* stage = smem + wave * (QB * 32 * C::ROWB);
  auto swz_out = [](int row) { return row & (C::UNITS - 1); };
  TS* outg = (TS*)a.out_states;
  const int64_t slot_elems = (int64_t)a.B * a.q_len * HD;
  const int64_t pt = part >= 0 ? (int64_t)(task - a.n_main) * a.split_f + part : 0;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = pair_sum(l[qb]);
    const int64_t row = row0 + qb * 32 + lr;
    if (row < a.q_len) {
      const float inv = lt > 0.f ? 1.0f / lt : 0.f;
      const float lse = lt > 0.f ? (m[qb] + __builtin_amdgcn_logf(lt)) * kLn2 : -INFINITY;
      if (part < 0) {
        if constexpr (sizeof(TS) == 2) {
          unsigned char* srow = stage + (qb * 32 + lr) * C::ROWB;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              f32x4 x;
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
              const int unit = (4 * db + r4) ^ swz_out(qb * 32 + lr);
              const int half = g ^ ((lr >> 4) & 1);
              *(bf16x4*)(srow + unit * 16 + 8 * half) = __builtin_convertvector(x, bf16x4);
            }
        } else {
          TS* dst = outg + (int64_t)slot * slot_elems + ((int64_t)b * a.q_len + row) * HD + (int64_t)h * D + 4 * g;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              f32x4 x;
#pragma unroll
              for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
              store4(dst + db * 32 + 8 * r4, x);
            }
        }
        if (g == 0) a.lse_states[(((int64_t)slot * a.B + b) * a.H + h) * a.q_len + row] = lse;
      } else {
        const int64_t rl = row - (int64_t)qt * C::BM;
        float* dst = a.part_out + (pt * C::BM + rl) * D + 4 * g;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            f32x4 x;
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = o[qb][db][4 * r4 + e] * inv;
            store4(dst + db * 32 + 8 * r4, x);
          }
        if (g == 0) a.part_lse[pt * C::BM + rl] = lse;
      }
    }
  }
  if constexpr (sizeof(TS) == 2) {
    if (part < 0) {
      const int ld_row = lane / C::UNITS, ld_unit = lane % C::UNITS;
      TS* dst0 = outg + (int64_t)slot * slot_elems + (int64_t)b * a.q_len * HD + (int64_t)h * D + ld_unit * 8;
#pragma unroll
      for (int i = 0; i < QB * 32 / C::ROWS_PER_LOAD; ++i) {
        const int row = i * C::ROWS_PER_LOAD + ld_row;
        if (row0 + row < a.q_len) {
          bf16x8 x = *(const bf16x8*)(stage + row * C::ROWB + ((ld_unit ^ swz_out(row)) * 16));
          if ((row >> 4) & 1) x = __builtin_shufflevector(x, x, 4, 5, 6, 7, 0, 1, 2, 3);
          *(bf16x8*)(dst0 + (row0 + row) * HD) = x;
        }
      }
    }
  }
}

// Composes the split_f partial states of every split task (Eq. composition
// over its key ranges) into the task's rows of its slot.  One thread per 8
// elements of a row.
template <int D, int BM, typename TS>
__global__ __launch_bounds__(256) void attn_split_fixup_kernel(const AttnArgs a) {
  constexpr int CPR = D / 8;
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= (int64_t)a.n_split * BM * CPR) return;
  const int ch = (int)(c % CPR);
  const int64_t rr = c / CPR;
  const int rl = (int)(rr % BM);
  const int t = (int)(rr / BM);
  int task = a.n_main + t;
  const int qt = task % a.q_tiles;
  task /= a.q_tiles;
  const int h = task % a.H;
  task /= a.H;
  const int b = task % a.B;
  const int sel = task / a.B;
  const int64_t row = (int64_t)qt * BM + rl;
  if (row >= a.q_len) return;
  const int f = a.split_f;
  const int64_t p0 = (int64_t)t * f;
  float lv[kMaxSplit];
  float mx = -INFINITY;
#pragma unroll
  for (int p = 0; p < kMaxSplit; ++p) {
    lv[p] = p < f ? a.part_lse[(p0 + p) * BM + rl] : -INFINITY;
    mx = fmaxf(mx, lv[p]);
  }
  float tot = 0.f;
#pragma unroll
  for (int p = 0; p < kMaxSplit; ++p) {
    lv[p] = mx == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((lv[p] - mx) * 1.4426950408889634f);
    tot += lv[p];
  }
  const float inv = tot > 0.f ? 1.0f / tot : 0.f;
  f32x4 acc0 = f32x4{}, acc1 = f32x4{};
#pragma unroll
  for (int p = 0; p < kMaxSplit; ++p) {
    if (p < f) {
      const float* src = a.part_out + ((p0 + p) * BM + rl) * D + ch * 8;
      const float w = lv[p] * inv;
      acc0 += w * *(const f32x4*)src;
      acc1 += w * *(const f32x4*)(src + 4);
    }
  }
  const int slot = a.slot[sel];
  const int64_t HD = (int64_t)a.H * D;
  TS* dst = (TS*)a.out_states + (int64_t)slot * a.B * a.q_len * HD + ((int64_t)b * a.q_len + row) * HD +
            (int64_t)h * D + ch * 8;
  store4(dst, acc0);
  store4(dst + 4, acc1);
  if (ch == 0)
    a.lse_states[(((int64_t)slot * a.B + b) * a.H + h) * a.q_len + row] =
        tot > 0.f ? mx + __builtin_amdgcn_logf(tot) * kLn2 : -INFINITY;
}

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Zeroes the queue counters of a balanced launch (a kernel, not a memset, so
// that the launch sequence can be captured in a graph).
__global__ __launch_bounds__(64) void attn_queue_reset_kernel(int* queue) {
  if (threadIdx.x < kQueueInts) queue[threadIdx.x] = 0;
}

// Dynamic share of the balanced launch: the last DITANGO_DYN_ROUNDS rounds of
// resident workgroups of every XCD's range are claimed from the queues.
#ifndef DITANGO_DYN_ROUNDS
#define DITANGO_DYN_ROUNDS 2
#endif

// Launch plan of one bf16 launch: resident workgroup slots on the current
// device, the tail split factor and number of split tasks, and the workspace
// bytes (queue counters, partial OUT in float32, partial LSE).
struct Plan {
  int64_t slots = 0;
  int f = 1;
  int64_t n_split = 0;
  size_t split_bytes = 0;   // partial states
  size_t bytes = 0;         // kQueueBytes + split_bytes (0: nothing launched)
};

// A kernel of the launch below: the compiled form (any tile configuration)
// or the hand-scheduled D=128 form.  Each names its function, workgroup
// size, query rows per workgroup and dynamic LDS.
template <int D, int QB, int NW, int BN, int NBUF, int WPE, bool SEQ, typename TS>
struct CompiledKernel {
  using C = Cfg<D, QB, NW, BN, NBUF>;
  static constexpr int Dim = D, NT = C::NT, BM = C::BM, KEYS = BN;
  static constexpr size_t LDS = C::LDS_BYTES;
  static const void* fn() { return (const void*)attn_bf16_kernel<D, QB, NW, BN, NBUF, WPE, SEQ, TS>; }
  static void launch(dim3 grid, hipStream_t s, const AttnArgs& a) {
    hipLaunchKernelGGL((attn_bf16_kernel<D, QB, NW, BN, NBUF, WPE, SEQ, TS>), grid, dim3(NT), LDS, s, a);
  }
};

template <int D, typename TS>
struct AsmKernel {
  using C = AsmCfg<D>;
  static constexpr int Dim = D, NT = C::NT, BM = C::BM, KEYS = C::BN;
  static constexpr size_t LDS = C::LDS_BYTES;
  static const void* fn() { return (const void*)attn_bf16_asm_kernel<D, TS>; }
  static void launch(dim3 grid, hipStream_t s, const AttnArgs& a) {
    hipLaunchKernelGGL((attn_bf16_asm_kernel<D, TS>), grid, dim3(NT), LDS, s, a);
  }
};

template <class K>
hipError_t set_lds() {
  static const hipError_t attr = hipFuncSetAttribute(K::fn(), hipFuncAttributeMaxDynamicSharedMemorySize, (int)K::LDS);
  return attr;
}

template <class K>
hipError_t plan_cfg(const AttnArgs& a, Plan* p) {
  hipError_t e = set_lds<K>();
  if (e != hipSuccess) return e;
  *p = Plan{};
  const int64_t nblk = (a.q_len + K::BM - 1) / K::BM * a.H * a.B * a.n_sel;
  if (nblk <= 0) return hipSuccess;
  int dev = 0, cus = 0, occ = 0;
  e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, K::fn(), K::NT, K::LDS);
  if (e != hipSuccess) return e;
  p->slots = (int64_t)cus * (occ > 0 ? occ : 1);
  p->bytes = kQueueBytes;
  // the split tasks are the launch's last ones: tiles of the last selected partition
  const int64_t tiles = ((int64_t)a.kv_len[a.n_sel - 1] + K::KEYS - 1) / K::KEYS;
  const int f = plan_tail_split(nblk, p->slots, tiles);
  if (f <= 1) return hipSuccess;
  p->f = f;
  p->n_split = nblk % p->slots;
  p->split_bytes = align256((size_t)p->n_split * f * K::BM * K::Dim * sizeof(float)) +
                   align256((size_t)p->n_split * f * K::BM * sizeof(float));
  p->bytes += p->split_bytes;
  return hipSuccess;
}

template <class K, typename TS>
hipError_t launch_cfg(const AttnArgs& a0, void* ws, size_t ws_bytes, hipStream_t s) {
  constexpr int D = K::Dim;
  Plan p;
  const bool queued = ws != nullptr && ws_bytes >= kQueueBytes;
  if (queued) {
    const hipError_t e = plan_cfg<K>(a0, &p);
    if (e != hipSuccess) return e;
  } else {
    const hipError_t e = set_lds<K>();
    if (e != hipSuccess) return e;
  }
  AttnArgs a = a0;
  a.q_tiles = (int)((a.q_len + K::BM - 1) / K::BM);
  const int64_t nblk = (int64_t)a.q_tiles * a.H * a.B * a.n_sel;
  if (nblk <= 0) return hipSuccess;
  if (nblk + (int64_t)kMaxSplit * p.n_split + p.slots > 0x7fffffff) return hipErrorInvalidConfiguration;
  a.n_main = (int)nblk;
  a.n_split = 0;
  a.split_f = 1;
  a.n_static = (int)nblk;
  a.queue = nullptr;
  int64_t grid = nblk;
  if (queued) {
    a.queue = (int*)ws;
    if (p.f > 1 && ws_bytes >= p.bytes) {
      a.n_main = (int)(nblk - p.n_split);
      a.n_split = (int)p.n_split;
      a.split_f = p.f;
      a.part_out = (float*)((char*)ws + kQueueBytes);
      a.part_lse = (float*)((char*)a.part_out + align256((size_t)p.n_split * p.f * K::BM * D * sizeof(float)));
    }
    // static share: the first positions of every XCD queue, all but its
    // last DITANGO_DYN_ROUNDS rounds and at least the first round (which
    // starts at once and gains nothing from claiming); as many extra
    // workgroups as dynamic units, up to one round, let the faster XCDs
    // take units from the slower ones' queues
    const int64_t per_xcd = p.slots / 8 > 0 ? p.slots / 8 : 1;
    const int64_t n_tail = (int64_t)a.n_split * a.split_f;
    int64_t min_len = INT64_MAX;
    for (int x = 0; x < 8; ++x) {
      const int64_t len = (a.n_main >> 3) + (x < (a.n_main & 7) ? 1 : 0) + (n_tail >> 3) + (x < (n_tail & 7) ? 1 : 0);
      min_len = len < min_len ? len : min_len;
    }
    int64_t st = min_len - DITANGO_DYN_ROUNDS * per_xcd;
    const int64_t first = min_len < per_xcd ? min_len : per_xcd;
    st = st > first ? st : first;
    const int64_t n_units = (int64_t)a.n_main + n_tail;
    const int64_t n_dyn = n_units - 8 * st;
    a.n_static = (int)(8 * st);
    grid = n_units + (n_dyn < p.slots ? n_dyn : p.slots);
    if (n_dyn > 0) {
      hipLaunchKernelGGL(attn_queue_reset_kernel, dim3(1), dim3(64), 0, s, a.queue);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  K::launch(dim3((unsigned)grid), s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split == 0) return e;
  const int64_t chunks = (int64_t)a.n_split * K::BM * (D / 8);
  hipLaunchKernelGGL((attn_split_fixup_kernel<D, K::BM, TS>), dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0,
                     s, a);
  return hipGetLastError();
}

// The hand-scheduled loops bound their tile loads with 32-bit buffer
// descriptors: every selected partition's bytes for one head must stay
// below 2^31.
inline bool asm_fits(const AttnArgs& a, int D) {
  const int64_t row_bytes = (int64_t)a.H * D * 2;
  for (int j = 0; j < a.n_sel; ++j)
    if ((int64_t)a.kv_len[j] * row_bytes >= ((int64_t)1 << 31)) return false;
  return true;
}

// Which D=64 kernel a launch runs.  At D=64 the softmax's VALU work per MFMA
// doubles and the hand-scheduled form gains little per tile (4 % at the
// 118,800-token, 48-head shape), while its 256-row query tiles make more
// tasks than the compiled kernel's 384-row ones: a launch that the compiled
// kernel runs in one round can take two (the 16,384-token, 12-head reuse
// launch: 288 tasks on 256 CUs against 216, 66.6 against 56 us).  So the
// hand-scheduled kernel runs only launches of at least four rounds.
inline bool d64_use_asm(const AttnArgs& a) {
  if (!asm_fits(a, 64)) return false;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return false;
  const int64_t tasks = (a.q_len + AsmCfg<64>::BM - 1) / AsmCfg<64>::BM * a.H * a.B * a.n_sel;
  return tasks >= 4 * (int64_t)cus;
}

}  // namespace

// Tile configuration per head dim: query blocks per wave, waves per
// workgroup, keys per tile, K/V ring size, minimum waves per SIMD, and the
// loop form (pipelined, or tile by tile).  D=128: 8 waves, two per SIMD,
// pipelined (256 VGPRs).  D=64: 12 waves, three per SIMD, 96-key tiles, tile
// by tile (166 VGPRs): the softmax VALU work per MFMA doubles at D=64, and a
// third wave per SIMD hides more of it than software pipelining does.
// Overridable at build time for tuning sweeps.
#ifndef DITANGO_D128_CFG
#define DITANGO_D128_CFG 1, 8, 64, 2, 2, false
#endif
#ifndef DITANGO_D64_CFG
#define DITANGO_D64_CFG 1, 12, 96, 2, 3, true
#endif
// Both head dims run the hand-scheduled kernel (attn_bf16_asm_kernel) unless
// built with DITANGO_ASM=0, or a partition is too long for its 32-bit
// tile-load bounds, or (D=64) the launch is short (d64_use_asm).
#ifndef DITANGO_ASM
#define DITANGO_ASM 1
#endif

hipError_t launch_attn_bf16_ws(const AttnArgs& a, int D, bool state_f32, void* ws, size_t ws_bytes,
                               hipStream_t s) {
  if (D == 128) {
#if DITANGO_ASM
    if (asm_fits(a, 128))
      return state_f32 ? launch_cfg<AsmKernel<128, float>, float>(a, ws, ws_bytes, s)
                       : launch_cfg<AsmKernel<128, __bf16>, __bf16>(a, ws, ws_bytes, s);
#endif
    return state_f32 ? launch_cfg<CompiledKernel<128, DITANGO_D128_CFG, float>, float>(a, ws, ws_bytes, s)
                     : launch_cfg<CompiledKernel<128, DITANGO_D128_CFG, __bf16>, __bf16>(a, ws, ws_bytes, s);
  }
  if (D == 64) {
#if DITANGO_ASM
    if (d64_use_asm(a))
      return state_f32 ? launch_cfg<AsmKernel<64, float>, float>(a, ws, ws_bytes, s)
                       : launch_cfg<AsmKernel<64, __bf16>, __bf16>(a, ws, ws_bytes, s);
#endif
    return state_f32 ? launch_cfg<CompiledKernel<64, DITANGO_D64_CFG, float>, float>(a, ws, ws_bytes, s)
                     : launch_cfg<CompiledKernel<64, DITANGO_D64_CFG, __bf16>, __bf16>(a, ws, ws_bytes, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attn_bf16(const AttnArgs& a, int D, bool state_f32, hipStream_t s) {
  return launch_attn_bf16_ws(a, D, state_f32, nullptr, 0, s);
}

hipError_t attn_bf16_ws_bytes(const AttnArgs& a, int D, size_t* bytes) {
  Plan p;
  *bytes = 0;
  // the plan depends on the kernel's occupancy, which the state type does
  // not change; the bf16-state instantiation is queried
  hipError_t e = hipErrorInvalidValue;
#if DITANGO_ASM
  if (D == 128 && asm_fits(a, 128))
    e = plan_cfg<AsmKernel<128, __bf16>>(a, &p);
  else if (D == 64 && d64_use_asm(a))
    e = plan_cfg<AsmKernel<64, __bf16>>(a, &p);
  else
#endif
  if (D == 128)
    e = plan_cfg<CompiledKernel<128, DITANGO_D128_CFG, __bf16>>(a, &p);
  else if (D == 64)
    e = plan_cfg<CompiledKernel<64, DITANGO_D64_CFG, __bf16>>(a, &p);
  if (e == hipSuccess) *bytes = p.bytes;
  return e;
}

}  // namespace ditango

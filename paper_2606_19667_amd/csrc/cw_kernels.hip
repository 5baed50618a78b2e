// Device half of libcw for gfx950 (MI355X): suffix KV append and suffix
// prefill attention over a paged, prefix-cached KV store.
//
// Paper Sec. 1 and 2.1: with a reused prefix of P cached tokens, only the S
// suffix tokens are prefilled; they attend causally over themselves and fully
// over the prefix, whose K/V the engine keeps in fixed-size blocks.
//
// Attention kernel design (one workgroup = 8 wavefronts, two per SIMD = one tile):
//  * A tile is (request r, KV head g, a run of T suffix rows); its 256 MFMA
//    rows pack the G = Hq/Hkv query heads of g over T = 256/G positions, so
//    every K/V byte staged in LDS serves all heads of the group.
//  * Each wave owns 32 packed rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16: in the 32x32 accumulator layout a lane then
//    holds one query column and 16 keys, so row max / sum need one exchange
//    with lane ^ 32 and the softmax state is lane-local.
//  * O^T = V^T P^T uses the packed probabilities directly as the B operand;
//    the cache keeps each V block transposed, so V operands are plain reads.
//  * K/V steps of 64 keys (4 blocks) are copied from the cache into a ring of
//    three LDS stages by load-to-LDS instructions, two to three steps ahead.
//  * Softmax in fp32 and base 2 with a lazily moved base; only steps that
//    cross the causal diagonal apply the mask; keys past the prompt end are
//    zero-filled so stale cache bytes never reach the result.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <string>
#include <type_traits>

#include "cw_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kBs = cw::kBlockSize;
constexpr int kKv = cw::kKvTile;

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bfloat16 (round to nearest even) in one dword, low first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// ---------------------------------------------------------------------------
// KV append. The unit of work is one block of suffix rows: request r
// contributes ceil(S_r / 16) units, unit j covering suffix rows 16 j ..
// min(16 j + 16, S_r) - 1, which (P_r being a multiple of 16) fill slots
// 0 .. of a single cache block. One workgroup per unit finds its (request,
// unit) with a wave-wide prefix sum over the per-request unit counts, copies
// the K rows ([slot][d] in the cache, contiguous 16-byte chunks) and writes V
// transposed ([d][slot]) by 8 x 8 register transposes: 16-byte stores per
// 8-slot half row, one element per slot where a partial block ends.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, u32x4* __restrict__ k_cache,
    uint16_t* __restrict__ v_cache, const int32_t* __restrict__ bt, int bt_stride,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ plen, int batch, int hkv, int D,
    int num_blocks) {
  __shared__ int s_unit[2];
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int b = blockIdx.x;
    int base = 0, rr = -1, jb = 0;
    for (int r0 = 0; r0 < batch; r0 += 64) {
      const int r = r0 + tid;
      const int n = r < batch ? (cu[r + 1] - cu[r] + kBs - 1) / kBs : 0;
      int x = n;   // inclusive prefix sum of n over the lanes
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (tid >= off) x += y;
      }
      const uint64_t hit = __ballot(base + x - n <= b && b < base + x);
      if (hit) {
        const int l = __ffsll(static_cast<unsigned long long>(hit)) - 1;
        rr = r0 + l;
        jb = b - base - __shfl(x - n, l);
        break;
      }
      base += __shfl(x, 63);
    }
    if (tid == 0) {
      s_unit[0] = rr;
      s_unit[1] = jb;
    }
  }
  __syncthreads();
  const int r = s_unit[0];
  if (r < 0) return;
  const int j0 = kBs * s_unit[1];
  const int cu0 = cu[r];
  const int nv = min(kBs, cu[r + 1] - cu0 - j0);
  const int t0 = plen[r] + j0;
  const int blk = bt[int64_t(r) * bt_stride + t0 / kBs];
  if (nv <= 0 || blk < 0 || blk >= num_blocks) return;

  const int nch = D / 8;   // 16-byte chunks per row and head
  const int64_t src0 = int64_t(cu0 + j0) * hkv * nch;
  // K: source chunk c = (slot, head, chunk) -> cache [blk][head][slot][chunk].
  // A thread issues all loads of a batch before its stores.
  u32x4* kd = k_cache + int64_t(blk) * hkv * kBs * nch;
  const int nk = nv * hkv * nch;
  constexpr int kBatch = 8;
  for (int c0 = tid; c0 < nk; c0 += kThreads * kBatch) {
    u32x4 kr[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) kr[i] = k_new[src0 + min(c0 + i * kThreads, nk - 1)];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int c = c0 + i * kThreads;
      if (c < nk) {
        const int ch = c & (nch - 1);
        const int rest = c / nch;
        kd[((rest % hkv) * kBs + rest / hkv) * nch + ch] = kr[i];
      }
    }
  }
  // V: the cache holds each block transposed, [blk][head][d][slot]. A task is
  // (head, 8 values of d, 8 slots): it loads the 8 slots' 16-byte chunks,
  // transposes the 8 x 8 block of bfloat16 in registers (v_perm) and stores 8
  // rows of 8 slots. Slots past the unit's rows are neither read (the row index
  // is clamped) nor written.
  uint16_t* vd = v_cache + int64_t(blk) * hkv * D * kBs;
  const int ntask = hkv * nch * 2;
  for (int u = tid; u < ntask; u += kThreads) {
    const int sh = u & 1;              // slots 8 sh .. 8 sh + 7
    const int dc = (u >> 1) % nch;     // d = 8 dc .. 8 dc + 7
    const int h = (u >> 1) / nch;
    const int nvs = min(8, nv - 8 * sh);   // valid slots of this task
    if (nvs <= 0) continue;
    uint32_t rw[8][4];                 // rw[k][j]: slot 8 sh + k, d pair j
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int slot = min(8 * sh + k, nv - 1);
      const u32x4 x = v_new[src0 + (int64_t(slot) * hkv + h) * nch + dc];
#pragma unroll
      for (int j = 0; j < 4; ++j) rw[k][j] = x[j];
    }
    uint16_t* dst = vd + (int64_t(h) * D + 8 * dc) * kBs + 8 * sh;
#pragma unroll
    for (int e = 0; e < 8; ++e) {      // output row d = 8 dc + e: 8 slots
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;   // high or low halves
      uint32_t o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = __builtin_amdgcn_perm(rw[2 * k + 1][e >> 1], rw[2 * k][e >> 1], sel);
      if (nvs == 8) {
        *reinterpret_cast<u32x4*>(dst + e * kBs) = u32x4{o[0], o[1], o[2], o[3]};
      } else {
        for (int k = 0; k < nvs; ++k) dst[e * kBs + k] = uint16_t(o[k >> 1] >> (16 * (k & 1)));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Suffix prefill attention.
//
// Work split: one workgroup = 8 wavefronts (two per SIMD) = one tile of 256
// packed query rows; wave w owns query columns 32 w .. 32 w + 31 and walks the
// tile's keys in steps of 64.
//
// Per wave the step loop is software-pipelined so that matrix and vector work
// of different steps overlap inside one instruction stream:
//   step j:  S(j+1) = K(j+1) Q^T  (16 MFMAs)  ||  P(j) = exp2(S(j))  (VALU)
//            O^T += V(j)^T P(j)^T (16 MFMAs)  ||  mask + row max of S(j+1)
//
// K/V staging: LDS holds three stages of (K, V) for one 64-key step. The
// cache blocks are copied into LDS by the LDS-direct loads (global_load_lds),
// which need no registers: wave w moves K (w even) or V (w odd) of block w / 2
// of a step, K three steps and V two steps ahead of their use, and waits for
// its copies of the step after next only at the end of the following step, so
// each copy has two steps to land. A block that is missing or reaches past the
// prompt end goes through registers instead and is zero-filled, so stale cache
// bytes never meet a zero probability. One barrier ends each step.
//
// Softmax in base 2 with lazy rescaling. Q is pre-multiplied by
// softmax_scale * log2(e) (rounded to bf16), and each S accumulator starts
// from -m, the running exponent base, so the MFMA result is already the
// exponent s - m. The base moves only when a row's step maximum exceeds it by
// more than 8 (a factor 256), and then O and l are rescaled once; probabilities
// therefore stay below 256 and the fp32 sums cannot overflow.
//
// LDS layouts (per stage). A load-to-LDS instruction writes 64 x 16 bytes
// contiguously in lane order, so swizzles are applied on the global side
// (each lane fetches the 16 bytes that belong at its LDS slot).
//  * K: row-major [key][d] (RB bytes per row); 16-byte chunk c of row r is
//    stored at c ^ kswz(r), which puts the 16 rows of every operand read phase
//    on distinct banks.
//  * V: the cache holds each block transposed, [d][slot]; LDS keeps that per
//    block ([block][d][16 keys], 32-byte rows) with the two 16-byte halves of
//    row d swapped when bit 3 of d is set (conflict-free operand reads).
//  * Key order: the PV MFMA's B operand is the score accumulator itself. In
//    the 32x32 accumulator, lane half u, register e holds row
//    8 (e / 4) + 4 u + e % 4. Reading K row pi(i) into A row i, with pi
//    swapping bits 2 and 3 of i, makes that register hold key
//    16 (e / 8) + 8 u + e % 8 (plus 32 per 32-key half), so for the 16-key
//    slice kk of the PV product lane half u holds keys 16 kk + 8 u .. + 7 in
//    order: block kk, half u of a V^T row, one 16-byte read.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

// The attention kernel orders its cache copies against its LDS reads itself,
// with explicit vmcnt waits and workgroup barriers. Its two memory helpers are
// asm statements so that the compiler does not add waits of its own: a
// load-to-LDS copy it can see makes it put a vmcnt(0) before LDS reads it
// cannot tell apart from the copy's target, and a register load it can see may
// be waited for with vmcnt(0) far from its use. Either drains every copy in
// flight. The compiler's own vmcnt waits only become more conservative for
// memory operations it does not see.

// 16 bytes through registers, waited for at once (every older memory operation
// of the wave completes with it). Used only for blocks that are not whole.
__device__ __forceinline__ u32x4 load16_now(const void* src) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(src) : "memory");
  return v;
}

// One load-to-LDS copy: lane l's 16 bytes at src land at dst + 16 l. M0 holds
// the LDS address (one wait state between writing M0 and the copy).
__device__ __forceinline__ void copy16_to_lds(const void* src, lds_void_t* dst) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst))) : "memory");
}

constexpr int kAttnWaves = 8;
constexpr int kAttnThreads = 64 * kAttnWaves;
static_assert(kAttnWaves * 32 == cw::kTileRows, "one 32-column MFMA block per wave");
constexpr int kStages = 3;

template <int D>
struct AttnGeom {
  static constexpr int RB = 2 * D;              // bytes per K row
  static constexpr int NC = D / 8;              // 16-byte chunks per K row
  static constexpr int KTILE = kKv * RB;        // K of one step
  static constexpr int BLK = D * 2 * kBs;       // one V^T block (D rows of 16 keys)
  static constexpr int VTILE = (kKv / kBs) * BLK;
  static constexpr int STAGE = KTILE + VTILE;
  static constexpr int RPL = 1024 / RB;         // K rows per 1 KB copy
  static constexpr int LPW = kBs * RB / 1024;   // 1 KB copies per block and tensor
  static constexpr int KS = D / 16;             // MFMA k-steps over D
  static constexpr int DT = D / 32;             // 32-row output tiles over D
  // chunk swizzle of K row r (rows of 256 bytes: 16 chunks; of 128 bytes: 8)
  __device__ static int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
};

constexpr float kLazy = 8.0f;   // rescale when a score exceeds the base by 2^8

// s_waitcnt immediates (gfx9 encoding): vmcnt(n) with lgkmcnt(0), expcnt untouched.
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 15) | (7 << 4) | ((n >> 4) << 14); }

// x * c rounded to bfloat16, for the 8 bfloat16 values of one Q fragment.
__device__ __forceinline__ bf16x8 scale_bf16x8(u32x4 raw, float c) {
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    o[j] = pack_bf16x2(__uint_as_float(raw[j] << 16) * c, __uint_as_float(raw[j] & 0xFFFF0000u) * c);
  return __builtin_bit_cast(bf16x8, u32x4{o[0], o[1], o[2], o[3]});
}

// SPLIT: the key range of each tile is divided into num_splits runs of whole
// steps processed by separate workgroups (workgroup s * num_tiles + i takes run s
// of plan entry i); each writes, for its rows, the attention over its keys only:
// O normalised in fp32 to part_o[s][row][d] and the base-2 log-sum-exp of the
// scaled scores to part_lse[s][row] (row = suffix row * Hq + head), -inf when
// no key of the run is visible. lse_merge_kernel combines the runs.
template <int D, bool SPLIT>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void suffix_prefill_attn_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
                                const uint16_t* __restrict__ vc, const int32_t* __restrict__ bt,
                                int bt_stride, const int32_t* __restrict__ cu,
                                const int32_t* __restrict__ plen, const int4* __restrict__ plan,
                                int batch, int hq, int hkv, int group, int per_tile, int num_blocks,
                                float c_log2, uint16_t* __restrict__ out, int num_splits, int num_tiles,
                                int64_t part_rows, float* __restrict__ part_o, float* __restrict__ part_lse) {
  using G = AttnGeom<D>;
  constexpr int KS = G::KS, DT = G::DT, RB = G::RB, NC = G::NC, LPW = G::LPW, RPL = G::RPL;
  constexpr int KTILE = G::KTILE, BLK = G::BLK, STAGE = G::STAGE;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * STAGE];

  const int tile = SPLIT ? int(blockIdx.x % unsigned(num_tiles)) : int(blockIdx.x);
  const int split = SPLIT ? int(blockIdx.x / unsigned(num_tiles)) : 0;
  const int4 item = plan[tile];
  const int r = item.x, g = item.y, row0 = item.z;
  if (r < 0 || r >= batch || g < 0 || g >= hkv) return;
  const int cu0 = cu[r];
  const int S = cu[r + 1] - cu0;
  const int P = plen[r];
  if (row0 < 0 || row0 >= S) return;
  const int L = P + S;
  const int nvalid = min(per_tile, S - row0);
  const int kv_end = P + row0 + nvalid;
  const int ntiles = (kv_end + kKv - 1) / kKv;
  // this workgroup's steps: tbeg .. tbeg + nsteps - 1 of the tile's key range
  int tbeg = 0, nsteps = ntiles;
  if (SPLIT) {
    const int per = (ntiles + num_splits - 1) / num_splits;
    tbeg = split * per;
    nsteps = max(0, min(ntiles, tbeg + per) - tbeg);
  }
  // local steps 0 .. n_full - 1 are visible to every row of the tile (no mask)
  const int n_full = max(0, min(nsteps, (P + row0 + 1) / kKv - tbeg));
  const int nblk = (L + kBs - 1) / kBs;
  const int32_t* btr = bt + int64_t(r) * bt_stride;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // This lane's query column.
  const int m = wave * 32 + l32;
  const int hh = m / per_tile;
  const int pos = m - hh * per_tile;
  const bool row_ok = (hh < group) && (pos < nvalid);
  const int qpos = P + row0 + pos;  // keys 0 .. qpos are visible
  const int64_t qrow = int64_t(cu0) + row0 + pos;
  const int head = g * group + hh;

  if (SPLIT && nsteps == 0) {   // no key of this run: an empty part
    if (row_ok) {
      const int64_t prow = int64_t(split) * part_rows + qrow * hq + head;
      float* po = part_o + prow * D;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq)
          *reinterpret_cast<f32x4*>(po + t * 32 + gq * 8 + half * 4) = f32x4{0.f, 0.f, 0.f, 0.f};
      if (half == 0) part_lse[prow] = -INFINITY;
    }
    return;
  }

  bf16x8 qf[KS];
  if (row_ok) {
    const u32x4* qp = reinterpret_cast<const u32x4*>(q + (qrow * hq + head) * D);
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = scale_bf16x8(qp[2 * s + half], c_log2);
  } else {
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
  }

  // ---- staging role of this wave: tensor (K or V) of block slot bs of a step
  const int bs = wave >> 1;
  const bool is_v = (wave & 1) != 0;
  const int ahead = is_v ? 2 : 3;   // step j copies the step j + ahead
  const uint16_t* const cache = is_v ? vc : kc;
  // Per-lane source offset inside a block (bytes) and LDS destination inside a
  // stage of copy i (the destination of lane l is dst + 16 l).
  int src_off[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    if (is_v) {
      const int d = 32 * i + (lane >> 1);
      src_off[i] = d * 32 + (((lane & 1) ^ ((lane >> 4) & 1)) << 4);
    } else {
      const int row = RPL * i + lane / NC;   // row inside the block
      src_off[i] = row * RB + (((lane % NC) ^ G::kswz(row)) << 4);
    }
  }
  const int dst0 = is_v ? KTILE + bs * BLK : bs * kBs * RB;
  // Physical block of logical block lb, or -1 past the prompt / outside the
  // pool; the table index is clamped into the request's row (always in bounds).
  auto block_id = [&](int lb) __attribute__((always_inline)) -> int {
    // read through the constant address space: a scalar load (a vector load
    // would be waited for with vmcnt, which also waits for the copies)
    const int b = reinterpret_cast<const __attribute__((address_space(4))) int32_t*>(
        reinterpret_cast<uintptr_t>(btr))[min(lb, nblk - 1)];
    return (lb < nblk && b >= 0 && b < num_blocks) ? b : -1;
  };
  // Stages step t's block of this wave into stage st; returns whether it used
  // the load-to-LDS path (whose completion the caller then waits for).
  auto stage_block = [&](int t, int b, int st) __attribute__((always_inline)) -> bool {
    const int key0 = (tbeg + t) * kKv + bs * kBs;
    const uint8_t* src = reinterpret_cast<const uint8_t*>(cache) +
                         (int64_t(b < 0 ? 0 : b) * hkv + g) * (kBs * RB);
    uint8_t* dst = lds + st * STAGE + dst0;
    if (b >= 0 && key0 + kBs <= L) {   // wave-uniform: the whole block is valid
#pragma unroll
      for (int i = 0; i < LPW; ++i)
        copy16_to_lds(src + src_off[i], (lds_void_t*)(dst + i * 1024));
      return true;
    }
    const u32x4 zero{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      u32x4 v = zero;
      if (b >= 0) v = load16_now(src + src_off[i]);
      if (is_v) {
        // keys key0 + 8 h .. + 7 of row d, h the logical half this lane holds
        const int h8 = 8 * ((lane & 1) ^ ((lane >> 4) & 1));
        const int vn = b < 0 ? 0 : min(8, max(0, L - key0 - h8));
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = 2 * j + 1 < vn ? v[j] : (2 * j < vn ? (v[j] & 0xFFFFu) : 0u);
      } else {
        const bool ok = b >= 0 && key0 + RPL * i + lane / NC < L;
        v = ok ? v : zero;
      }
      *reinterpret_cast<u32x4*>(dst + i * 1024 + lane * 16) = v;
    }
    return false;
  };
  // End of a step: this wave's copies for the next step have landed (the LPW
  // copies issued in this step may still be in flight, when `keep` says that
  // nothing else went to memory after them), LDS writes are done, then the
  // workgroup barrier. The empty asm statements keep the compiler from moving
  // memory accesses across the barrier.
  auto step_barrier = [&](bool keep) __attribute__((always_inline)) {
    if (keep) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(LPW));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // ---- per-lane LDS read offsets (relative to a stage)
  // K operand: row 32 h + pi(l32), logical chunk 2 s + half.
  const int k_row = (l32 & ~12) | ((l32 & 4) << 1) | ((l32 & 8) >> 1);
  int k_off[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) k_off[s] = k_row * RB + (((2 * s + half) ^ G::kswz(k_row)) << 4);
  // V operand: block kk, row d = 32 t + l32, logical half = half.
  const int v_off = KTILE + l32 * 32 + ((half ^ ((l32 >> 3) & 1)) << 4);

  // ---- the four pieces of a step
  // S^T = K Q^T for one stage, accumulators starting from c0.
  auto qk = [&](const uint8_t* st, const f32x16& c0, f32x16 (&sc)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(st + k_off[s] + h * 32 * RB));
        sc[h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], s == 0 ? c0 : sc[h], 0, 0, 0);
      }
  };
  // Causal mask of the step starting at key k0.
  auto mask = [&](f32x16 (&sc)[2], int k0) __attribute__((always_inline)) {
    // key of element e of half h is h 32 + (e / 8) 16 + half 8 + e % 8; the
    // lane term moves to the limit so that the per-element terms stay immediates
    const int lim = qpos - k0 - half * 8;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (h * 32 + (e >> 3) * 16 + (e & 7) > lim) sc[h][e] = -INFINITY;
  };
  // Maximum of the row over the step's 64 keys (this lane's 32 and lane ^ 32's).
  auto rowmax = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) -> float {
    float a = fmaxf(fmaxf(sc[0][0], sc[0][1]), sc[0][2]);
    float b = fmaxf(fmaxf(sc[1][0], sc[1][1]), sc[1][2]);
#pragma unroll
    for (int e = 3; e < 15; e += 2) {
      a = fmaxf(fmaxf(a, sc[0][e]), sc[0][e + 1]);
      b = fmaxf(fmaxf(b, sc[1][e]), sc[1][e + 1]);
    }
    a = fmaxf(fmaxf(a, sc[0][15]), sc[1][15]);
    a = fmaxf(a, b);
    return fmaxf(a, __shfl_xor(a, 32));
  };
  float l_run = 0.f;   // this lane's partial row sum (its 32 keys per step)
  const bf16x2 ones{(__bf16)1.0f, (__bf16)1.0f};
  // Probabilities 2^(s - m) as the PV B operand; adds their sum to l_run.
  auto probs = [&](const f32x16 (&sc)[2], bf16x8 (&pb)[4]) __attribute__((always_inline)) {
    float ls[2] = {0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int h = kk >> 1, e0 = (kk & 1) * 8;
      uint32_t w[4];   // a scalar array: bit casts of ext-vector elements are not used
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        w[j] = pack_bf16x2(__builtin_amdgcn_exp2f(sc[h][e0 + 2 * j]),
                           __builtin_amdgcn_exp2f(sc[h][e0 + 2 * j + 1]));
        ls[kk & 1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[j]), ones, ls[kk & 1], false);
      }
      pb[kk] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
    l_run += ls[0] + ls[1];
  };
  f32x16 oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) oacc[t] = f32x16{};
  // O^T += V^T P^T for one stage.
  auto pv = [&](const uint8_t* st, const bf16x8 (&pb)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(st + v_off + kk * BLK + t * 1024));
        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kk], oacc[t], 0, 0, 0);
      }
  };

  // ---- prologue: stage steps 0 and 1 (and K of step 2); S(0) with the exact
  // row maximum as base
  {
    const int n0 = min(nsteps, ahead);
    for (int t = 0; t < n0; ++t) stage_block(t, block_id((tbeg + t) * (kKv / kBs) + bs), t);
  }
  // block copied in step 0
  int bnext = ahead < nsteps ? block_id((tbeg + ahead) * (kKv / kBs) + bs) : -1;
  step_barrier(false);
  f32x16 sa[2], sb[2];
  qk(lds, f32x16{}, sa);
  if (n_full == 0) mask(sa, tbeg * kKv);
  f32x16 mneg;   // -m in every element: the start of each S accumulator
  {
    // Finite when the run's first step has a visible key for this row (always
    // so for the first run: key 0 is visible to every row). A row that sees no
    // key of the run's first step sees none of its later steps either (they
    // hold higher keys), so any base serves it.
    float m0 = rowmax(sa);
    if (SPLIT && m0 == -INFINITY) m0 = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) sa[h] -= m0;
#pragma unroll
    for (int e = 0; e < 16; ++e) mneg[e] = -m0;
  }
  float mx = 0.f;   // row maximum of the current S (relative to the base)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();   // K of stage 0 is refilled during step 0
  asm volatile("" ::: "memory");

  // Moves the base up by the step maximum when it exceeds the base by kLazy.
  auto rebase = [&](f32x16 (&sc)[2]) __attribute__((always_inline)) {
    const bool grow = mx > kLazy;
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float delta = grow ? mx : 0.f;
      const float alpha = __builtin_amdgcn_exp2f(-delta);
#pragma unroll
      for (int h = 0; h < 2; ++h) sc[h] -= delta;
      mneg -= delta;
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t) oacc[t] *= alpha;
    }
  };
  // Step j < nsteps - 1: current S in sc, next S into sn. Stage of local step
  // t is t % 3; this wave copies step j + ahead into stage (j + ahead) % 3.
  auto step = [&](auto maskc, int j, f32x16 (&sc)[2], f32x16 (&sn)[2]) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(maskc)::value;
    rebase(sc);
    const int tc = j + ahead;
    bool issued = false;
    if (tc < nsteps) issued = stage_block(tc, bnext, tc % kStages);
    bnext = tc + 1 < nsteps ? block_id((tbeg + tc + 1) * (kKv / kBs) + bs) : -1;
    bf16x8 pb[4];
    qk(lds + ((j + 1) % kStages) * STAGE, mneg, sn);
    probs(sc, pb);
    pv(lds + (j % kStages) * STAGE, pb);
    if (MASK) mask(sn, (tbeg + j + 1) * kKv);
    mx = rowmax(sn);
    // masked steps may spill registers to scratch memory: wait for everything
    step_barrier(issued && !MASK);
  };
  using F = std::false_type;
  using T = std::true_type;
  const int last = nsteps - 1;
  int j = 0;
  // steps whose successor needs no mask, then the rest; two per iteration so
  // the S buffers alternate without copies
  auto run = [&](auto maskc, int end) __attribute__((always_inline)) {
    for (; j + 1 < end; j += 2) {
      step(maskc, j, sa, sb);
      step(maskc, j + 1, sb, sa);
    }
    if (j < end) {
      step(maskc, j, sa, sb);
#pragma unroll
      for (int h = 0; h < 2; ++h) sa[h] = sb[h];
      ++j;
    }
  };
  run(F{}, min(n_full - 1, last));
  run(T{}, last);
  {
    rebase(sa);
    bf16x8 pb[4];
    probs(sa, pb);
    pv(lds + (last % kStages) * STAGE, pb);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  if constexpr (SPLIT) {
    const int64_t prow = int64_t(split) * part_rows + qrow * hq + head;
    float* po = part_o + prow * D;
    const bool any = l_tot > 0.f;
    const float inv = any ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq)
        *reinterpret_cast<f32x4*>(po + t * 32 + gq * 8 + half * 4) =
            f32x4{oacc[t][gq * 4 + 0] * inv, oacc[t][gq * 4 + 1] * inv, oacc[t][gq * 4 + 2] * inv,
                  oacc[t][gq * 4 + 3] * inv};
    // base-2 log-sum-exp of the scaled scores: the base plus log2 of the sum
    if (half == 0) part_lse[prow] = any ? -mneg[0] + __log2f(l_tot) : -INFINITY;
    return;
  }
  const float inv = 1.f / l_tot;
  uint16_t* op = out + (qrow * hq + head) * D;
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int d = t * 32 + gq * 8 + half * 4;
      const u32x2 w{pack_bf16x2(oacc[t][gq * 4 + 0] * inv, oacc[t][gq * 4 + 1] * inv),
                    pack_bf16x2(oacc[t][gq * 4 + 2] * inv, oacc[t][gq * 4 + 3] * inv)};
      *reinterpret_cast<u32x2*>(op + d) = w;
    }
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge of attention results over disjoint key sets: for each row,
// out = sum_p 2^(lse_p - M) o_p / sum_p 2^(lse_p - M), M = max_p lse_p, where o_p
// is part p's normalised output and lse_p its base-2 log-sum-exp (-inf for a
// part with no keys). One thread per row and 8 consecutive elements.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void lse_merge_kernel(const float* __restrict__ part_o,
                                                             const float* __restrict__ part_lse,
                                                             int num_parts, int64_t rows, int d,
                                                             uint16_t* __restrict__ out) {
  const int per_row = d / 8;
  const int64_t u = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (u >= rows * per_row) return;
  const int64_t row = u / per_row;
  const int c = int(u - row * per_row);
  float m = -INFINITY;
  for (int p = 0; p < num_parts; ++p) m = fmaxf(m, part_lse[int64_t(p) * rows + row]);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  if (m != -INFINITY) {
    for (int p = 0; p < num_parts; ++p) {
      const float lp = part_lse[int64_t(p) * rows + row];
      if (lp == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(lp - m);
      wsum += w;
      const f32x4* src = reinterpret_cast<const f32x4*>(part_o + (int64_t(p) * rows + row) * d + c * 8);
      const f32x4 a = src[0], b = src[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[e] = fmaf(w, a[e], acc[e]);
        acc[4 + e] = fmaf(w, b[e], acc[4 + e]);
      }
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const u32x4 o{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)};
  *reinterpret_cast<u32x4*>(out + row * d + c * 8) = o;
}

cw_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return cw::fail(CW_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  return cw::ok();
}

}  // namespace

extern "C" cw_status cw_kv_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                                  const int32_t* block_table, int32_t bt_stride,
                                  const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                  const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                  int32_t batch, int32_t num_kv_heads, int32_t head_dim,
                                  int32_t block_size, int32_t num_blocks, void* stream) {
  if (!k_new || !v_new || !k_cache || !v_cache || !block_table || !cu_suffix_dev || !prefix_len_dev)
    return cw::fail(CW_EINVAL, "kv_append: a required pointer is NULL");
  if (num_kv_heads < 1) return cw::fail(CW_EINVAL, "kv_append: num_kv_heads must be >= 1");
  if (num_blocks < 1) return cw::fail(CW_EINVAL, "kv_append: num_blocks must be >= 1");
  if (head_dim != 64 && head_dim != 128) return cw::fail(CW_EUNSUPPORTED, "kv_append: head_dim must be 64 or 128");
  if (block_size != kBs) return cw::fail(CW_EUNSUPPORTED, "kv_append: block_size must be 16");
  int64_t rows = 0;
  cw_status st = cw::check_batch(cu_suffix_host, prefix_len_host, batch, block_size, bt_stride, &rows);
  if (st != CW_OK) return st;
  if (rows == 0) return cw::ok();
  int64_t units = 0;   // blocks of suffix rows
  for (int32_t r = 0; r < batch; ++r) units += (cu_suffix_host[r + 1] - cu_suffix_host[r] + kBs - 1) / kBs;
  if (units > INT32_MAX) return cw::fail(CW_EUNSUPPORTED, "kv_append: batch too large");
  hipLaunchKernelGGL(kv_append_kernel, dim3(unsigned(units)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(k_new),
                     static_cast<const u32x4*>(v_new), static_cast<u32x4*>(k_cache),
                     static_cast<uint16_t*>(v_cache), block_table, bt_stride, cu_suffix_dev,
                     prefix_len_dev, batch, num_kv_heads, head_dim, num_blocks);
  return check_launch("kv_append launch");
}

namespace {

// Checks shared by both attention entry points; fills the launch geometry.
struct AttnShape {
  int group = 0, per_tile = 0;
  int64_t rows = 0;
};
cw_status check_attn(const char* what, const void* q, const void* k_cache, const void* v_cache,
                     const int32_t* block_table, int32_t bt_stride, const int32_t* cu_suffix_dev,
                     const int32_t* prefix_len_dev, const int32_t* cu_suffix_host,
                     const int32_t* prefix_len_host, int32_t batch, int32_t num_q_heads,
                     int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t num_blocks,
                     float softmax_scale, const int32_t* plan_dev, int32_t num_tiles, const void* out,
                     AttnShape* shape) {
  const std::string w(what);
  if (!q || !k_cache || !v_cache || !block_table || !cu_suffix_dev || !prefix_len_dev || !out)
    return cw::fail(CW_EINVAL, w + ": a required pointer is NULL");
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0)
    return cw::fail(CW_EINVAL, w + ": num_q_heads must be a positive multiple of num_kv_heads");
  if (num_blocks < 1) return cw::fail(CW_EINVAL, w + ": num_blocks must be >= 1");
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    return cw::fail(CW_EINVAL, w + ": softmax_scale must be finite and positive");
  if (head_dim != 64 && head_dim != 128) return cw::fail(CW_EUNSUPPORTED, w + ": head_dim must be 64 or 128");
  if (block_size != kBs) return cw::fail(CW_EUNSUPPORTED, w + ": block_size must be 16");
  shape->group = num_q_heads / num_kv_heads;
  if (shape->group > cw::kMaxGroup)
    return cw::fail(CW_EUNSUPPORTED, w + ": more than 128 query heads per KV head");
  cw_status st = cw::check_batch(cu_suffix_host, prefix_len_host, batch, block_size, bt_stride, &shape->rows);
  if (st != CW_OK) return st;
  shape->per_tile = cw::tile_positions(shape->group);
  const int64_t need = cw::count_tiles(cu_suffix_host, batch, num_kv_heads, shape->per_tile);
  if (num_tiles < need || int64_t(num_tiles) > need * cw::kNumXcd)
    return cw::fail(CW_EINVAL, w + ": num_tiles " + std::to_string(num_tiles) + " does not match the batch (" +
                                   std::to_string(need) + " tiles)");
  if (num_tiles > 0 && !plan_dev) return cw::fail(CW_EINVAL, w + ": plan_dev is required");
  return CW_OK;
}

template <bool SPLIT>
void launch_attn(int head_dim, unsigned grid, hipStream_t s, const void* q, const void* k_cache,
                 const void* v_cache, const int32_t* block_table, int32_t bt_stride,
                 const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev, const int32_t* plan_dev,
                 int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, const AttnShape& sh,
                 int32_t num_blocks, float softmax_scale, void* out, int num_splits, int num_tiles,
                 int64_t part_rows, float* part_o, float* part_lse) {
  const float c_log2 = softmax_scale * 1.4426950408889634f;
  auto* qp = static_cast<const uint16_t*>(q);
  auto* kp = static_cast<const uint16_t*>(k_cache);
  auto* vp = static_cast<const uint16_t*>(v_cache);
  auto* pp = reinterpret_cast<const int4*>(plan_dev);
  auto* op = static_cast<uint16_t*>(out);
  if (head_dim == 128)
    hipLaunchKernelGGL((suffix_prefill_attn_kernel<128, SPLIT>), dim3(grid), dim3(kAttnThreads), 0, s, qp, kp, vp,
                       block_table, bt_stride, cu_suffix_dev, prefix_len_dev, pp, batch, num_q_heads,
                       num_kv_heads, sh.group, sh.per_tile, num_blocks, c_log2, op, num_splits, num_tiles,
                       part_rows, part_o, part_lse);
  else
    hipLaunchKernelGGL((suffix_prefill_attn_kernel<64, SPLIT>), dim3(grid), dim3(kAttnThreads), 0, s, qp, kp, vp,
                       block_table, bt_stride, cu_suffix_dev, prefix_len_dev, pp, batch, num_q_heads,
                       num_kv_heads, sh.group, sh.per_tile, num_blocks, c_log2, op, num_splits, num_tiles,
                       part_rows, part_o, part_lse);
}

constexpr int kMaxSplits = 64;

// Workspace of the split path: part_o [splits][rows][D] fp32, then part_lse
// [splits][rows] fp32 at a 256-byte aligned offset.
int64_t split_lse_offset(int64_t part_rows, int head_dim, int num_splits) {
  return (int64_t(num_splits) * part_rows * head_dim * 4 + 255) / 256 * 256;
}

cw_status launch_merge(const float* part_o, const float* part_lse, int num_parts, int64_t rows, int head_dim,
                       void* out, hipStream_t s) {
  const int64_t units = rows * (head_dim / 8);
  const int64_t grid = (units + kThreads - 1) / kThreads;
  if (grid > INT32_MAX) return cw::fail(CW_EUNSUPPORTED, "lse_merge: too many rows");
  if (grid == 0) return cw::ok();
  hipLaunchKernelGGL(lse_merge_kernel, dim3(unsigned(grid)), dim3(kThreads), 0, s, part_o, part_lse, num_parts,
                     rows, head_dim, static_cast<uint16_t*>(out));
  return check_launch("lse_merge launch");
}

}  // namespace

extern "C" cw_status cw_suffix_prefill_attn(const void* q, const void* k_cache, const void* v_cache,
                                            const int32_t* block_table, int32_t bt_stride,
                                            const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                            const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                            int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                            int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                            float softmax_scale, const int32_t* plan_dev,
                                            int32_t num_tiles, void* out, void* stream) {
  AttnShape sh;
  cw_status st = check_attn("suffix_prefill_attn", q, k_cache, v_cache, block_table, bt_stride, cu_suffix_dev,
                            prefix_len_dev, cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads,
                            head_dim, block_size, num_blocks, softmax_scale, plan_dev, num_tiles, out, &sh);
  if (st != CW_OK) return st;
  if (sh.rows == 0 || num_tiles == 0) return cw::ok();
  launch_attn<false>(head_dim, unsigned(num_tiles), static_cast<hipStream_t>(stream), q, k_cache, v_cache,
                     block_table, bt_stride, cu_suffix_dev, prefix_len_dev, plan_dev, batch, num_q_heads,
                     num_kv_heads, sh, num_blocks, softmax_scale, out, 1, num_tiles, 0, nullptr, nullptr);
  return check_launch("suffix_prefill_attn launch");
}

extern "C" int64_t cw_suffix_prefill_split_workspace_bytes(int64_t total_rows, int32_t num_q_heads,
                                                           int32_t head_dim, int32_t num_splits) {
  if (total_rows < 0 || num_q_heads < 1 || (head_dim != 64 && head_dim != 128) || num_splits < 1 ||
      num_splits > kMaxSplits)
    return cw::fail(CW_EINVAL, "suffix_prefill_split_workspace_bytes: invalid argument");
  const int64_t part_rows = total_rows * num_q_heads;
  return split_lse_offset(part_rows, head_dim, num_splits) + int64_t(num_splits) * part_rows * 4;
}

extern "C" cw_status cw_suffix_prefill_attn_split(const void* q, const void* k_cache, const void* v_cache,
                                                  const int32_t* block_table, int32_t bt_stride,
                                                  const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                                  const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                                  int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                                  int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                                  float softmax_scale, const int32_t* plan_dev,
                                                  int32_t num_tiles, int32_t num_splits, void* workspace,
                                                  int64_t workspace_bytes, void* out, void* stream) {
  AttnShape sh;
  cw_status st = check_attn("suffix_prefill_attn_split", q, k_cache, v_cache, block_table, bt_stride,
                            cu_suffix_dev, prefix_len_dev, cu_suffix_host, prefix_len_host, batch, num_q_heads,
                            num_kv_heads, head_dim, block_size, num_blocks, softmax_scale, plan_dev, num_tiles,
                            out, &sh);
  if (st != CW_OK) return st;
  if (num_splits < 1 || num_splits > kMaxSplits)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn_split: num_splits must be in [1, 64]");
  if (int64_t(num_tiles) * num_splits > INT32_MAX)
    return cw::fail(CW_EUNSUPPORTED, "suffix_prefill_attn_split: too many workgroups");
  const int64_t part_rows = sh.rows * num_q_heads;
  const int64_t need = cw_suffix_prefill_split_workspace_bytes(sh.rows, num_q_heads, head_dim, num_splits);
  if (!workspace || workspace_bytes < need)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn_split: workspace must hold " + std::to_string(need) + " bytes");
  if (sh.rows == 0 || num_tiles == 0) return cw::ok();
  auto* s = static_cast<hipStream_t>(stream);
  auto* part_o = static_cast<float*>(workspace);
  auto* part_lse = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                            split_lse_offset(part_rows, head_dim, num_splits));
  launch_attn<true>(head_dim, unsigned(int64_t(num_tiles) * num_splits), s, q, k_cache, v_cache, block_table,
                    bt_stride, cu_suffix_dev, prefix_len_dev, plan_dev, batch, num_q_heads, num_kv_heads, sh,
                    num_blocks, softmax_scale, out, num_splits, num_tiles, part_rows, part_o, part_lse);
  st = check_launch("suffix_prefill_attn_split launch");
  if (st != CW_OK) return st;
  return launch_merge(part_o, part_lse, num_splits, part_rows, head_dim, out, s);
}

extern "C" cw_status cw_lse_merge(const void* partial_o, const void* partial_lse, int32_t num_parts,
                                  int64_t rows, int32_t head_dim, void* out, void* stream) {
  if (!partial_o || !partial_lse || !out) return cw::fail(CW_EINVAL, "lse_merge: a required pointer is NULL");
  if (num_parts < 1) return cw::fail(CW_EINVAL, "lse_merge: num_parts must be >= 1");
  if (rows < 0) return cw::fail(CW_EINVAL, "lse_merge: rows must be >= 0");
  if (head_dim < 8 || head_dim % 8 != 0 || head_dim > 1024)
    return cw::fail(CW_EUNSUPPORTED, "lse_merge: head_dim must be a multiple of 8 in [8, 1024]");
  return launch_merge(static_cast<const float*>(partial_o), static_cast<const float*>(partial_lse), num_parts,
                      rows, head_dim, out, static_cast<hipStream_t>(stream));
}

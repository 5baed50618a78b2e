// Device half of libcw for gfx950 (MI355X): suffix KV append and suffix
// prefill attention over a paged, prefix-cached KV store.
//
// Paper Sec. 1 and 2.1: with a reused prefix of P cached tokens, only the S
// suffix tokens are prefilled; they attend causally over themselves and fully
// over the prefix, whose K/V the engine keeps in fixed-size blocks.
//
// Attention kernel design (persistent workgroups of 8 wavefronts, two per SIMD):
//  * A plan entry is (request r, KV head g, a run of T suffix rows, a run of
//    64-key steps); its 256 MFMA rows pack the G = Hq/Hkv query heads of g
//    over T = 256/G positions, so every K/V byte staged in LDS serves all
//    heads of the group. Workgroup w runs entries w, w + grid, ...
//  * Each wave owns 32 packed rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16: in the 32x32 accumulator layout a lane then
//    holds one query column and 16 keys, so row max / sum need one exchange
//    with lane ^ 32 and the softmax state is lane-local.
//  * O^T = V^T P^T uses the packed probabilities directly as the B operand;
//    its V^T operand comes from token-major V by transposing LDS reads.
//  * K/V steps of 64 keys (4 blocks) are copied from the cache into a ring of
//    four LDS stages by load-to-LDS instructions three steps ahead, by a copy
//    cursor that runs across entry boundaries.
//  * Softmax in fp32 and base 2 with a lazily moved base; only steps that
//    cross the causal diagonal apply the mask; keys past the prompt end are
//    zero-filled so stale cache bytes never reach the result.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>
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
typedef short s16x4 __attribute__((ext_vector_type(4)));

// Two floats to two bfloat16 (round to nearest even) in one dword, low first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// ---------------------------------------------------------------------------
// KV append. The unit of work is one block of suffix rows: request r
// contributes ceil(S_r / 16) units, unit j covering suffix rows 16 j ..
// min(16 j + 16, S_r) - 1, which (P_r being a multiple of 16) fill slots
// 0 .. of a single cache block. One workgroup per unit finds its (request,
// unit) with a wave-wide prefix sum over the per-request unit counts and
// copies the K and V rows ([slot][d] in both caches) in 16-byte chunks.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, u32x4* __restrict__ k_cache,
    u32x4* __restrict__ v_cache, const int32_t* __restrict__ bt, int bt_stride,
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

  // Source chunk c = (slot, head, chunk) of either tensor goes to cache
  // [blk][head][slot][chunk]. A thread issues all loads of a batch (K and V)
  // before its stores.
  const int nch = D / 8;   // 16-byte chunks per row and head
  const int64_t src0 = int64_t(cu0 + j0) * hkv * nch;
  const int64_t dst0 = int64_t(blk) * hkv * kBs * nch;
  const int nk = nv * hkv * nch;
  constexpr int kBatch = 8;
  for (int c0 = tid; c0 < nk; c0 += kThreads * kBatch) {
    u32x4 kr[kBatch], vr[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int64_t c = src0 + min(c0 + i * kThreads, nk - 1);
      kr[i] = k_new[c];
      vr[i] = v_new[c];
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int c = c0 + i * kThreads;
      if (c < nk) {
        const int ch = c & (nch - 1);
        const int rest = c / nch;
        const int64_t o = dst0 + ((rest % hkv) * kBs + rest / hkv) * nch + ch;
        k_cache[o] = kr[i];
        v_cache[o] = vr[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Suffix prefill attention.
//
// Work: the host plan lists entries (request r, KV head g, a run of T suffix
// rows, a run of 64-key steps); 256 packed MFMA rows of an entry hold the
// G = Hq / Hkv query heads of g over T = 256 / G positions, so each K/V byte
// staged in LDS serves the whole group. The grid is persistent: workgroup w
// (8 wavefronts, two per SIMD) runs plan entries w, w + grid, w + 2 grid, ...
// until an entry with r < 0, so one workgroup per CU walks its whole queue.
//
// Staging. LDS holds a ring of four stages of one 64-key step each (K and V
// of 4 blocks). A copy cursor, independent of the entry being computed, walks
// the workgroup's queue three steps ahead of the computation and copies each
// step's blocks into ring position p % 4 with load-to-LDS instructions (no
// registers): wave w moves K (w even) or V (w odd) of block w / 2 of the step.
// Because the cursor crosses entry boundaries, the first steps of the next
// entry are already in LDS while the current entry ends. A block that is not
// whole (the prompt's partial last block) goes through registers and is
// zero-filled past the prompt end; a missing block (past the prompt, or an
// out-of-pool table entry) reads as zeros.
//
// Per wave the step loop is software-pipelined so that matrix and vector work
// of different steps overlap in one instruction stream:
//   step j:  S(j+1) = K(j+1) Q^T  (MFMA)  ||  P(j) = exp2(S(j)), row sums (VALU)
//            O^T += V(j)^T P(j)^T (MFMA)  ||  mask + row max of S(j+1)      (VALU)
// with the LDS operand reads of both products issued three MFMAs ahead.
//
// Each wave owns 32 packed rows (query columns) and computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16: in the 32x32 accumulator a lane then holds one
// query column and 16 keys, so the softmax state is lane-local and a row
// reduction needs one exchange with lane ^ 32 (v_permlane32_swap). O^T = V^T
// P^T uses the packed probabilities as the B operand; its A operand (8
// consecutive keys of one d per lane) comes from V rows staged token-major by
// two transposing LDS reads (ds_read_b64_tr_b16).
//
// Softmax in base 2 with lazy rescaling. Q is pre-multiplied by
// softmax_scale * log2(e) (rounded to bf16), and each S accumulator starts
// from -m, the running exponent base, so the MFMA result is already the
// exponent s - m. The base moves only when a row's step maximum exceeds it by
// more than 8 (a factor 256), and then O and l are rescaled once;
// probabilities therefore stay below 256 and the fp32 sums cannot overflow.
//
// LDS layouts. A load-to-LDS instruction writes 64 x 16 bytes contiguously in
// lane order, so swizzles are applied on the global side (each lane fetches
// the 16 bytes that belong at its LDS slot).
//  * K stages: each block of 16 keys chunk-major, [16-byte chunk c][key r]
//    at c 256 + r 16: the 16 keys a read phase takes sit on distinct banks,
//    and a lane's operand reads differ only by immediate offsets.
//  * V stages (after the four K stages): chunk-major like K, key r of chunk c
//    at slot r ^ 4 (c % 4): a transposing read takes 4 keys of 4 consecutive
//    chunks, which this swizzle puts on distinct banks.
//  * Key order: the PV MFMA's B operand is the score accumulator itself. In
//    the 32x32 accumulator, lane half u, register e holds row
//    8 (e / 4) + 4 u + e % 4. Reading K row pi(i) into A row i, with pi
//    swapping bits 2 and 3 of i, makes that register hold key
//    16 (e / 8) + 8 u + e % 8 (plus 32 per 32-key half), so for the 16-key
//    slice kk of the PV product lane half u holds keys 16 kk + 8 u .. + 7 in
//    order: block kk, keys 8 u .. + 7 of one d, two transposing reads.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(4))) int32_t cint32_t;

// The attention kernel orders its cache copies against its LDS reads itself,
// with explicit vmcnt waits and workgroup barriers. Its memory helpers are asm
// statements so that the compiler does not add waits of its own: a
// load-to-LDS copy it can see makes it put a vmcnt(0) before LDS reads it
// cannot tell apart from the copy's target. The compiler's own vmcnt waits
// only become more conservative for memory operations it does not see.

// 16 bytes through registers, waited for at once (every older memory operation
// of the wave completes with it). Used only for blocks that are not whole.
__device__ __forceinline__ u32x4 load16_now(const void* src) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(src) : "memory");
  return v;
}

// Loads whose completion the compiler does not track. The attention kernel
// mixes them with load-to-LDS copies it issues itself, which the compiler does
// not see either; a load the compiler tracks makes it wait for every copy in
// flight (vmcnt(0)) before the first use. The caller guarantees that a wait
// covering the load (a step barrier's vmcnt) comes before the first read of the
// result, and ties the read to that point with an empty asm statement.
__device__ __forceinline__ int32_t load_word_untracked(const int32_t* src) {
  int32_t v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(src));
  return v;
}
__device__ __forceinline__ u32x4 load16_untracked(const void* src) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(src));
  return v;
}

// A word at a wave-uniform address (SGPRs), completion untracked as above.
__device__ __forceinline__ int32_t load_word_untracked_s(const int32_t* base) {
  const uint64_t b = reinterpret_cast<uintptr_t>(base);
  const uint64_t bu = (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b >> 32)))) << 32) |
                      uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b))));
  int32_t v;
  asm volatile("global_load_dword %0, %1, %2" : "=v"(v) : "v"(0u), "s"(bu));
  return v;
}
// Two words (8-byte aligned) at a wave-uniform address, completion untracked.
__device__ __forceinline__ u32x2 load_pair_untracked_s(const int32_t* base) {
  const uint64_t b = reinterpret_cast<uintptr_t>(base);
  const uint64_t bu = (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b >> 32)))) << 32) |
                      uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b))));
  u32x2 v;
  asm volatile("global_load_dwordx2 %0, %1, %2" : "=v"(v) : "v"(0u), "s"(bu));
  return v;
}

// Brings the 128-byte line holding src (per lane) into L2 with a 4-byte
// load-to-LDS per lane into lds_addr + 4 l, an area whose bytes nothing reads;
// completion untracked as above.
__device__ __forceinline__ void touch_line(const void* src, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds_addr)) : "memory");
}

// One load-to-LDS copy: lane l's 16 bytes at base + off + 64 k land at
// lds + 16 l (k = 0 .. 3). base is wave-uniform (SGPRs), off a per-lane 32-bit
// offset; M0 holds the LDS address (one wait state between writing M0 and the
// copy). The instruction's immediate offset is not used for the 64 k: it would
// move the LDS destination as well.
// (The uniform operands go through readfirstlane: the values are wave-uniform,
// and this keeps them in SGPRs where the compiler cannot prove it.)
__device__ __forceinline__ void copy16_to_lds(const void* base, uint32_t off, uint32_t lds_addr, int k) {
  const uint64_t b = reinterpret_cast<uintptr_t>(base);
  // readfirstlane returns int: widen through uint32_t so the low half is not
  // sign-extended into the high half
  const uint64_t bu = (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b >> 32)))) << 32) |
                      uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(b))));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off + 64u * uint32_t(k)), "s"(bu), "s"(__builtin_amdgcn_readfirstlane(lds_addr)) : "memory");
}

constexpr int kAttnWaves = 8;
constexpr int kAttnThreads = 64 * kAttnWaves;
static_assert(kAttnWaves * 32 == cw::kTileRows, "one 32-column MFMA block per wave");
constexpr int kStages = 4;   // LDS ring positions
constexpr int kAhead = 3;    // the cursor copies a step this many steps before its use

template <int D>
struct AttnGeom {
  static constexpr int RB = 2 * D;              // bytes per K row
  static constexpr int KTILE = kKv * RB;        // K of one step
  static constexpr int BLK = kBs * RB;          // one V block (16 keys of D values)
  static constexpr int VTILE = (kKv / kBs) * BLK;
  static constexpr int KREG = kStages * KTILE;  // the V stages start here
  static constexpr int RING = KREG + kStages * VTILE;
  static constexpr int STAGING = 4096;          // per-wave area after the ring
  static constexpr int LDS = RING + kAttnWaves * STAGING;
  static constexpr int LPW = kBs * RB / 1024;   // 1 KB copies per block and tensor
  static constexpr int KS = D / 16;             // MFMA k-steps over D
  static constexpr int DT = D / 32;             // 32-row output tiles over D
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(32 * RB + (KS - 1) * 512 < 65536, "K read offsets are immediates");
  static_assert((kStages - 1) * VTILE + 3 * BLK + (DT - 1) * 1024 < 65536, "V read offsets are immediates");
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

// max(x of this lane, x of lane ^ 32)
__device__ __forceinline__ float max_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Plan layout shared with the host planner (words of int32).
constexpr int kPlanHeader = cw::kPlanHeaderWords;
constexpr int kEntryWords = cw::kPlanEntryWords;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* bt;     // block table; for FUSED the plan's table of (source, destination) pairs
  const int32_t* plan;   // device copy of the whole plan (header, then entries)
  const uint16_t* kn;    // FUSED: the suffix K / V rows [total_s, Hkv, D]
  const uint16_t* vn;
  uint16_t* kw;          // FUSED: the caches, written at the suffix blocks
  uint16_t* vw;
  uint16_t* out;
  float* part_o;         // split runs: normalised O per run, fp32
  float* part_lse;       // split runs: base-2 log-sum-exp per run
  int64_t part_rows;     // rows of one run's part: total_s * Hq
  int32_t bt_stride, hq, hkv, group, per_tile, num_blocks, num_entries;
  int32_t total_rows;    // FUSED: rows of k_new / v_new
  float c_log2;
  uint32_t fp_lo, fp_hi; // the batch fingerprint the host validated
};

// SPLIT: entries may cover only part of a tile's key range (the planner cuts
// each tile into num_splits runs of whole steps); an entry then writes, for its
// rows, the attention over its keys only: O normalised in fp32 to
// part_o[split][row][d] and the base-2 log-sum-exp of the scaled scores to
// part_lse[split][row] (row = suffix row * Hq + head), -inf when no key of the
// run is visible. lse_merge_kernel combines the runs.
//
// FUSED (unsplit only): the KV append happens inside the call. The table of
// the plan gives each logical block a source (a cache block, 16 rows of
// k_new / v_new, or nothing) and a destination: a block whose rows are this
// call's suffix rows is staged from k_new / v_new, and the entry whose query
// rows are those rows also writes them, from the LDS stage, into the block's
// place in the caches. No entry reads a cache block that the call writes.
template <int D, bool SPLIT, bool FUSED>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void suffix_prefill_attn_kernel(const AttnArgs a) {
  static_assert(!(SPLIT && FUSED), "the fused call is unsplit");
  using G = AttnGeom<D>;
  constexpr int KS = G::KS, DT = G::DT, RB = G::RB, LPW = G::LPW;
  constexpr int KTILE = G::KTILE, BLK = G::BLK, VTILE = G::VTILE, KREG = G::KREG;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[G::LDS];
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));

  cint32_t* plan = reinterpret_cast<cint32_t*>(reinterpret_cast<uintptr_t>(a.plan));
  // A plan whose header does not carry the fingerprint of the batch the host
  // validated is not this batch's plan: compute nothing.
  if (uint32_t(plan[cw::kHdrFpLo]) != a.fp_lo || uint32_t(plan[cw::kHdrFpHi]) != a.fp_hi) return;
  const int32_t* const ents = a.plan + kPlanHeader;
  const int grid = int(gridDim.x);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- staging role of this wave: tensor (K or V) of block slot bs of a step
  const int bs = wave >> 1;
  const bool is_v = (wave & 1) != 0;
  const uint8_t* const cache = reinterpret_cast<const uint8_t*>(is_v ? a.vc : a.kc);
  // bytes from one physical block of a tensor to the next (below 2^28: the
  // host refuses more than kMaxKvHeads KV heads), multiplied by a block ID as
  // two 32-bit values
  const uint32_t blk_bytes = uint32_t(a.hkv) * (kBs * RB);
  // Per-lane source offset inside a block and LDS destination of copy i
  // (relative to the wave's block slot in a stage; lane l lands at +16 l).
  // Both tensors are staged chunk-major: 16-byte chunk c of key row r of a
  // block at c 256 + r' 16, with r' = r for K and r' = r ^ 4 (c % 4) for V, so
  // copy i (chunks 4 i .. 4 i + 3) brings lane l the chunk 4 i + l / 16 of key
  // ckey (below).
  // ckey (below). Copy i adds 64 i (its immediate offset) to the lane's base:
  // off_c for a cache block (rows RB apart), off_n for rows of k_new / v_new
  // (rows Hkv RB apart).
  const int ckey = is_v ? ((lane & 15) ^ ((lane >> 4) << 2)) : (lane & 15);
  const uint32_t off_c = uint32_t(ckey * RB + ((lane >> 4) << 4));
  const uint32_t row_bytes = uint32_t(a.hkv) * RB;   // FUSED: from one k_new row to the next
  const uint32_t off_n = FUSED ? uint32_t(ckey) * row_bytes + uint32_t((lane >> 4) << 4) : 0u;
  const uint8_t* const fresh_base = reinterpret_cast<const uint8_t*>(is_v ? a.vn : a.kn);
  // FUSED: largest source index of a whole block: cache blocks (16 b) and
  // k_new / v_new rows (the host refuses pools of 2^27 blocks or more)
  const int cache_lim = 16 * a.num_blocks - 16;
  const int fresh_lim = a.total_rows - 16;
  // table words per logical block
  constexpr int TW = FUSED ? 2 : 1;
  // LDS address of this wave's block slot in ring position 0
  const uint32_t slot0 = lds0 + (is_v ? KREG + bs * BLK : bs * kBs * RB);
  const uint32_t stage_stride = is_v ? VTILE : KTILE;
  // This wave's area after the ring: output staging, and the target of loads
  // whose data nothing reads.
  const uint32_t own_area = lds0 + G::RING + wave * G::STAGING;

  // ---- copy cursor: the entry and step whose blocks this wave copies next.
  // Its state is wave-uniform. The words of the next entry the cursor enters
  // are prefetched into cdesc (lane l holds word l % 16), loaded when the
  // cursor enters the entry before it, so that a step that moves the cursor to
  // a new entry waits for no load.
  int ce = blockIdx.x;   // index of the entry whose words are in cdesc
  int c_left = 0;        // steps of the cursor's entry not yet issued
  int c_lb = 0;          // this wave's logical block at the cursor's step
  int c_whole = 0;       // logical blocks below this hold 16 keys of the prompt
  int c_last = 0;        // last logical block inside the prompt
  int c_L = 0;           // prompt length of the cursor's request
  int c_fast = 0;        // steps from the cursor's step that take the fast path of issue()
  const int32_t* c_row = a.bt;   // block-table row of the cursor's request
  const int32_t* c_ptr = a.bt;   // table word of this wave's block at the cursor's step
  const uint8_t* c_src = cache;  // this wave's tensor at the cursor's KV head
  int64_t c_delta = 0;   // FUSED: from c_src to this wave's tensor at that head in k_new / v_new
  bool cdone = false;
  auto entry_word_addr = [&](int e) __attribute__((always_inline)) -> const int32_t* {
    return ents + int64_t(min(e, a.num_entries - 1)) * kEntryWords + (lane & 15);
  };
  int32_t cdesc = load_word_untracked(entry_word_addr(ce));
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(cdesc) :: "memory");
  // Makes the entry whose words are in cdesc the cursor's entry and loads the
  // words of the one after it; ends the cursor at the end of the queue or at
  // an entry not written for this batch.
  auto cursor_take = [&]() __attribute__((always_inline)) {
    if (ce >= a.num_entries) { cdone = true; return; }
    const int r = __builtin_amdgcn_readlane(cdesc, cw::kEntR);
    const uint32_t tag = uint32_t(__builtin_amdgcn_readlane(cdesc, cw::kEntCheck));
    if (r < 0 || tag != cw::entry_tag(a.fp_lo, a.fp_hi, uint32_t(ce))) { cdone = true; return; }
    const int kb = __builtin_amdgcn_readlane(cdesc, cw::kEntKbeg);
    c_left = __builtin_amdgcn_readlane(cdesc, cw::kEntKend) - kb;
    c_lb = kb * (kKv / kBs) + bs;
    c_L = __builtin_amdgcn_readlane(cdesc, cw::kEntL);
    c_whole = c_L / kBs;
    c_last = (c_L + kBs - 1) / kBs - 1;
    c_row = a.bt + int64_t(r) * a.bt_stride * TW;
    c_ptr = c_row + c_lb * TW;
    const int cg = __builtin_amdgcn_readlane(cdesc, cw::kEntG);
    c_src = cache + int64_t(cg) * (kBs * RB);
    if constexpr (FUSED) c_delta = (fresh_base + int64_t(cg) * RB) - c_src;
    // Fast steps: not the entry's last (whose issue() enters the next entry),
    // the block whole (lb < c_whole) and the next step's table word inside
    // the prompt's blocks (lb + 4 <= c_last), so that it needs no clamp.
    const int lim = min(c_whole, c_last - (kKv / kBs - 1));
    c_fast = min(c_left - 1, max(0, (lim - c_lb + kKv / kBs - 1) / (kKv / kBs)));
    ce += grid;
    cdesc = load_word_untracked(entry_word_addr(ce));
  };
  // As cursor_take, skipping entries without steps (empty split runs): each
  // further entry first waits for the words its predecessor loaded (so every
  // path back to the reads passes that wait).
  auto cursor_enter = [&]() __attribute__((always_inline)) {
    cursor_take();
    if (!cdone && c_left == 0) {
      do {
        asm volatile("s_waitcnt vmcnt(0)" : "+v"(cdesc) :: "memory");
        cursor_take();
      } while (!cdone && c_left == 0);
    }
  };
  // Block-table word (FUSED: the table's pair) of this wave's block at the
  // cursor's step, loaded one step before its copies: issue() loads it before
  // its own copies, so the step barrier that follows (which leaves only those
  // copies in flight) completes it. The index is clamped into the prompt. Past
  // the last entry harmless words (the plan's first) are loaded.
  std::conditional_t<FUSED, u32x2, int32_t> bword{};
  auto load_bword = [&](const int32_t* w) __attribute__((always_inline)) {
    if constexpr (FUSED) bword = load_pair_untracked_s(w);
    else bword = load_word_untracked_s(w);
  };
  auto cursor_load = [&]() __attribute__((always_inline)) {
    c_ptr = c_row + min(c_lb, c_last) * TW;
    load_bword(cdone ? a.plan : c_ptr);
  };
  // FUSED: the destination word of the block each ring position holds (lane
  // p % 4), recorded when the block is copied, -1 when nothing is written.
  int32_t dring = -1;
  cursor_enter();
  cursor_load();
  // The copies of a step are spread over the step's MFMAs rather than issued
  // together: eight waves issuing all of theirs at once fill the load queue
  // and stall at the step start. issue() records where copy k goes; a copy of
  // a step without load-to-LDS copies rewrites this wave's own area with bytes
  // of block 0, which nothing reads (the step then waits for all).
  uint64_t cp_src = reinterpret_cast<uintptr_t>(cache);
  uint32_t cp_dst = own_area, cp_stride = 0, cp_off = off_c;
  auto copy_part = [&](int k) __attribute__((always_inline)) {
    copy16_to_lds(reinterpret_cast<const void*>(cp_src), cp_off, cp_dst + k * cp_stride, k);
  };
  // Copies the cursor's step into ring position p (now, or through copy_part
  // when `spread`) and advances the cursor. Returns whether load-to-LDS
  // copies of this wave are in flight (a block that is not whole is written
  // through registers and waited for at once). The table word it reads was
  // completed by the wait before this call.
  auto issue = [&](int p, bool spread) __attribute__((always_inline)) -> bool {
    asm volatile("" : "+v"(bword));
    int raw, dword = -1;
    if constexpr (FUSED) {
      raw = __builtin_amdgcn_readfirstlane(int(bword[0]));
      dword = __builtin_amdgcn_readfirstlane(int(bword[1]));
    } else {
      raw = __builtin_amdgcn_readfirstlane(bword);
    }
    const uint32_t dst = slot0 + uint32_t(p & (kStages - 1)) * stage_stride;
    if constexpr (!FUSED) {
      // fast path: a whole block inside the pool, the next word inside the
      // prompt's blocks, the cursor stays in its entry (c_fast > 0 implies
      // !cdone)
      if (c_fast > 0 && uint32_t(raw) < uint32_t(a.num_blocks)) {
        const uint8_t* src = c_src + uint64_t(uint32_t(raw)) * blk_bytes;
        --c_fast;
        --c_left;
        c_lb += kKv / kBs;
        c_ptr += kKv / kBs;
        load_bword(c_ptr);
        if (spread) {
          cp_src = reinterpret_cast<uintptr_t>(src);
          cp_dst = dst;
          cp_stride = 1024;
        } else {
#pragma unroll
          for (int i = 0; i < LPW; ++i) copy16_to_lds(src, off_c, dst + i * 1024, i);
        }
        return true;
      }
      cp_src = reinterpret_cast<uintptr_t>(cache);
      cp_dst = own_area;
      cp_stride = 0;
      if (cdone) return false;
      const int lb = c_lb, L = c_L;
      // physical block, or -1 past the prompt / outside the pool
      const int b = (lb <= c_last && uint32_t(raw) < uint32_t(a.num_blocks)) ? raw : -1;
      const bool whole = b >= 0 && lb < c_whole;
      const uint8_t* src = c_src + uint64_t(uint32_t(b < 0 ? 0 : b)) * blk_bytes;
      c_lb += kKv / kBs;
      c_fast = max(0, c_fast - 1);
      if (--c_left == 0) cursor_enter();
      cursor_load();
      if (whole) {   // wave-uniform: the whole block is valid
        if (spread) {
          cp_src = reinterpret_cast<uintptr_t>(src);
          cp_dst = dst;
          cp_stride = 1024;
        } else {
#pragma unroll
          for (int i = 0; i < LPW; ++i) copy16_to_lds(src, off_c, dst + i * 1024, i);
        }
        return true;
      }
      const int key0 = lb * kBs;
      const u32x4 zero{0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        // (a missing block loads block 0 and discards it, so that every path
        // through here waits for the memory operations issued before it)
        u32x4 v = load16_now(src + off_c + 64 * i);
        const bool ok = b >= 0 && key0 + ckey < L;
        v = ok ? v : zero;
        *reinterpret_cast<u32x4*>(lds + (dst - lds0) + i * 1024 + lane * 16) = v;
      }
      return false;
    } else {
      // The block's source: the cache block raw (FUSED: the word is 16 b for
      // cache block b, or 0x80000000 | R for rows R .. R + 15 of k_new / v_new,
      // both scaled by row_bytes; -1 or any other value out of range is no
      // block). `inb`: a whole block of that source lies inside its tensor.
      // (selects by masks of the word's sign: the compiler keeps them scalar)
      const int sgn = raw >> 31;   // -1 for rows of k_new / v_new, else 0
      const bool neg = sgn != 0;
      const uint32_t idx = uint32_t(raw) & 0x7FFFFFFFu;
      const bool inb = int(idx) <= cache_lim + (sgn & (fresh_lim - cache_lim));
      auto where = [&](uint32_t i) __attribute__((always_inline)) -> const uint8_t* {
        return c_src + (int64_t(sgn) & c_delta) + uint64_t(i) * row_bytes;
      };
      // fast path: a whole block, the next word inside the prompt's blocks, the
      // cursor stays in its entry (c_fast > 0 implies !cdone)
      if (c_fast > 0 && inb) {
        const uint8_t* src = where(idx);
        if constexpr (FUSED) dring = lane == (p & (kStages - 1)) ? dword : dring;
        --c_fast;
        --c_left;
        c_lb += kKv / kBs;
        c_ptr += (kKv / kBs) * TW;
        load_bword(c_ptr);
        const uint32_t off = neg ? off_n : off_c;
        if (spread) {
          cp_src = reinterpret_cast<uintptr_t>(src);
          cp_dst = dst;
          cp_stride = 1024;
          cp_off = off;
        } else {
  #pragma unroll
          for (int i = 0; i < LPW; ++i) copy16_to_lds(src, off, dst + i * 1024, i);
        }
        return true;
      }
      cp_src = reinterpret_cast<uintptr_t>(cache);
      cp_dst = own_area;
      cp_stride = 0;
      cp_off = off_c;
      if (cdone) {
        if constexpr (FUSED) dring = lane == (p & (kStages - 1)) ? -1 : dring;
        return false;
      }
      const int lb = c_lb, L = c_L;
      const int key0 = lb * kBs;
      // a block inside the prompt whose rows up to the prompt's end lie inside
      // the source tensor (a partial block of k_new / v_new rows is not read
      // past the prompt: the last request's end is the tensor's end)
      bool valid = lb <= c_last;
      if constexpr (FUSED) valid = valid && (neg ? int64_t(idx) + (L - 1 - key0) < a.total_rows : inb);
      else valid = valid && inb;
      const bool whole = valid && lb < c_whole;
      const uint8_t* src = where(valid ? idx : 0u);
      if constexpr (FUSED) dring = lane == (p & (kStages - 1)) ? (lb <= c_last ? dword : -1) : dring;
      c_lb += kKv / kBs;
      c_fast = max(0, c_fast - 1);
      if (--c_left == 0) cursor_enter();
      cursor_load();
      if (whole) {   // wave-uniform: the whole block is valid
        const uint32_t off = neg ? off_n : off_c;
        if (spread) {
          cp_src = reinterpret_cast<uintptr_t>(src);
          cp_dst = dst;
          cp_stride = 1024;
          cp_off = off;
        } else {
  #pragma unroll
          for (int i = 0; i < LPW; ++i) copy16_to_lds(src, off, dst + i * 1024, i);
        }
        return true;
      }
      const u32x4 zero{0, 0, 0, 0};
      const uint32_t off_p =
          (neg && valid) ? uint32_t(min(ckey, L - 1 - key0)) * row_bytes + uint32_t((lane >> 4) << 4) : off_c;
  #pragma unroll
      for (int i = 0; i < LPW; ++i) {
        // (a missing block loads block 0 and discards it, so that every path
        // through here waits for the memory operations issued before it)
        u32x4 v = load16_now(src + off_p + 64 * i);
        const bool ok = valid && key0 + ckey < L;
        v = ok ? v : zero;
        *reinterpret_cast<u32x4*>(lds + (dst - lds0) + i * 1024 + lane * 16) = v;
      }
      return false;
      }
  };
  // End of a step: this wave's copies for the next steps have landed (the
  // copies issued in this step may still be in flight when `keep` says that
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

  // ---- per-lane LDS read offsets (ring position 0; a position adds its stride)
  // K operand: key 32 h + pi(l32) (block 2 h + l32 / 16, row pi(l32) % 16),
  // chunk 2 s + half; in the chunk-major block layout that is the lane's base
  // plus h 32 RB + s 512.
  const int k_row = (l32 & ~12) | ((l32 & 4) << 1) | ((l32 & 8) >> 1);
  int k_off = (l32 >> 4) * (kBs * RB) + half * 256 + (k_row & 15) * 16;
  // V operand (transposing reads, two per operand): in each 16-lane group a
  // lane names 4 values of d of one key, and lane 4 q + s receives value s of
  // the 4 keys named by lanes q, q + 4, q + 8, q + 12. Lane j of group gq names
  // key 8 half + 4 rd + j / 4 of the block (rd: first or second read) and
  // d = 32 t + 16 (gq % 2) + 4 (j % 4), so lane l32 receives row d = 32 t + l32,
  // keys 8 half + 4 rd .. + 3: with both reads the operand of keys
  // 8 half .. + 7. In the swizzled chunk-major layout that is the lane's base
  // (chunk c % 4 = 2 (gq % 2) + (j % 4) / 2) plus t 1024 + kk BLK.
  const int vj = lane & 15, vpart = 2 * ((lane >> 4) & 1) + ((vj & 3) >> 1);
  int v_off0 = KREG + vpart * 256 + (((8 * half + (vj >> 2)) ^ (4 * vpart)) << 4) + 8 * (vj & 1);
  int v_off1 = KREG + vpart * 256 + (((8 * half + 4 + (vj >> 2)) ^ (4 * vpart)) << 4) + 8 * (vj & 1);
  // Hide the bases' known bits from the compiler: otherwise it rewrites
  // base + constant as base | constant, which it cannot fold into the LDS
  // instructions' offset field, and keeps one register per read instead.
  asm volatile("" : "+v"(k_off));
  asm volatile("" : "+v"(v_off0));
  asm volatile("" : "+v"(v_off1));
  auto rd16 = [&](int addr) __attribute__((always_inline)) -> bf16x8 {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(lds + addr));
  };
  auto rdtr = [&](int addr) __attribute__((always_inline)) -> u32x2 {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    auto* lp = (__attribute__((address_space(3))) uint8_t*)lds + addr;
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)lp));
  };

  // This lane's query column inside a tile: head hh of the group, position pos.
  const int m = wave * 32 + l32;
  const int hh = m / a.per_tile;
  const int pos = m - hh * a.per_tile;

  // Raw Q (bf16) of the entry to come, loaded before the first steps for the
  // first entry and during an entry's last step for the next one, so that an
  // entry starts without waiting for its queries.
  u32x4 qn[KS];
  // Plan entry words of the entry to come and of the one after it, one word
  // per lane: lane l holds word l % 16 of entry e (l % 32 < 16) or of entry
  // e + grid (l % 32 >= 16; past the last entry, the last entry's words).
  // Loaded with the queries, so that an entry starts without a scalar load.
  int32_t desc = 0;
  auto load_desc = [&](int e) __attribute__((always_inline)) {
    const int idx = min(e + ((lane >> 4) & 1) * grid, a.num_entries - 1);
    desc = load_word_untracked(ents + int64_t(idx) * kEntryWords + (lane & 15));
  };
  // word i of the entry (second = false) or of the one after it
  auto desc_word = [&](int32_t dw, bool second, int i) __attribute__((always_inline)) -> int {
    return __builtin_amdgcn_readlane(dw, (second ? 16 : 0) + i);
  };
  // This lane's Q row in the entry after the current one (`exists` false past
  // the last entry); row 0 of Q for a lane without a row or past the last
  // entry (the load stays inside Q and the entry discards the value).
  auto q_source = [&](int32_t dw, bool second, bool exists) __attribute__((always_inline)) -> const u32x4* {
    int64_t off = 0;
    if (exists) {
      const int r = desc_word(dw, second, cw::kEntR), nv = desc_word(dw, second, cw::kEntNvalid);
      const int64_t row = int64_t(desc_word(dw, second, cw::kEntQrow)) + pos;
      const int hd = desc_word(dw, second, cw::kEntG) * a.group + hh;
      off = (r >= 0 && hh < a.group && pos < nv) ? (row * a.hq + hd) * D : 0;
    }
    return reinterpret_cast<const u32x4*>(a.q + off);
  };
  auto load_q = [&](const u32x4* qp) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < KS; ++s) qn[s] = load16_untracked(qp + 2 * s + half);
  };
  load_desc(blockIdx.x);
  // the wait that completes the words (and the table word loaded before),
  // tied to the register that receives them
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(desc) :: "memory");
  load_q(q_source(desc, false, true));
  // the first call below reads the table word: complete since the wait above

  // ---- first steps of the queue
  int p = 0;   // ring position of the next step to compute
#pragma unroll
  for (int i = 0; i < kAhead; ++i) {
    // the next call reads the table word this one loaded: wait for it, leaving
    // the copies issued after it in flight
    if (issue(i, false)) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(LPW));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // Output rows of the staged read-back (unsplit kernel): the lanes reading
  // staged row rr hold column m' = 32 wave + rr of the tile, i.e. head m' / T
  // and position m' % T (T = a.per_tile; the quotient by a multiply, exact for
  // m' < 256).
  const uint32_t tdiv = (65536u + uint32_t(a.per_tile) - 1) / uint32_t(a.per_tile);

  for (int e = blockIdx.x; e < a.num_entries; e += grid) {
    // the words landed before the previous entry's last step barrier (or the
    // first steps' wait)
    asm volatile("" : "+v"(desc));
    const int32_t dw = desc;
    // the end of the queue, or an entry that is not the one the planner wrote
    if (desc_word(dw, false, cw::kEntR) < 0 ||
        uint32_t(desc_word(dw, false, cw::kEntCheck)) != cw::entry_tag(a.fp_lo, a.fp_hi, uint32_t(e)))
      break;
    // where the next entry's Q comes from
    const u32x4* q_next = q_source(dw, true, e + grid < a.num_entries);
    const int g = desc_word(dw, false, cw::kEntG), row0 = desc_word(dw, false, cw::kEntRow0);
    const int nvalid = desc_word(dw, false, cw::kEntNvalid), P = desc_word(dw, false, cw::kEntP);
    const int qrow0 = desc_word(dw, false, cw::kEntQrow);
    const int kbeg = desc_word(dw, false, cw::kEntKbeg);
    const int nsteps = desc_word(dw, false, cw::kEntKend) - kbeg;
    // steps [0, n_full) are visible to every row of the entry (no mask)
    const int n_full = desc_word(dw, false, cw::kEntNfull);
    const int split = SPLIT ? desc_word(dw, false, cw::kEntSplit) : 0;

    const bool row_ok = (hh < a.group) && (pos < nvalid);
    const int qpos = P + row0 + pos;  // keys 0 .. qpos are visible
    const int64_t qrow = int64_t(qrow0) + pos;
    const int head = g * a.group + hh;

    if (SPLIT && nsteps == 0) {   // no key of this run: an empty part
      if (row_ok) {
        const int64_t prow = int64_t(split) * a.part_rows + qrow * a.hq + head;
        float* po = a.part_o + prow * D;
#pragma unroll
        for (int t = 0; t < DT; ++t)
#pragma unroll
          for (int gq = 0; gq < 4; ++gq)
            *reinterpret_cast<f32x4*>(po + t * 32 + gq * 8 + half * 4) = f32x4{0.f, 0.f, 0.f, 0.f};
        if (half == 0) a.part_lse[prow] = -INFINITY;
      }
      // the next entry's Q and words, waited for here (this entry has no
      // last step)
      load_q(q_next);
      load_desc(e + grid);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      continue;
    }

    bf16x8 qf[KS];
    {
      // qn landed before the last step barrier (or the first steps' wait, or
      // an empty run's wait)
#pragma unroll
      for (int s = 0; s < KS; ++s) asm volatile("" : "+v"(qn[s]));
#pragma unroll
      for (int s = 0; s < KS; ++s)
        qf[s] = row_ok ? scale_bf16x8(qn[s], a.c_log2) : __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
    }

    // Causal mask of the step starting at key k0: element e of accumulator h
    // holds key k0 + 32 h + (e / 8) 16 + half 8 + e % 8; the lane term moves to
    // the limit so that the per-element terms stay immediates.
    // (each element is pinned after its select: otherwise the compiler keeps
    // all 32 compare results live as lane masks in scalar registers)
    auto mask = [&](f32x16 (&sc)[2], int k0) __attribute__((always_inline)) {
      const int lim = qpos - k0 - half * 8;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e2 = 0; e2 < 16; ++e2) {
          if (h * 32 + (e2 >> 3) * 16 + (e2 & 7) > lim) sc[h][e2] = -INFINITY;
          asm volatile("" : "+v"(sc[h][e2]));
        }
    };
    // Maximum of the row over a step's 64 keys (this lane's 32 and lane ^ 32's).
    auto rowmax = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) -> float {
      float x = fmaxf(fmaxf(sc[0][0], sc[0][1]), sc[0][2]);
      float y = fmaxf(fmaxf(sc[1][0], sc[1][1]), sc[1][2]);
#pragma unroll
      for (int e2 = 3; e2 < 15; e2 += 2) {
        x = fmaxf(fmaxf(x, sc[0][e2]), sc[0][e2 + 1]);
        y = fmaxf(fmaxf(y, sc[1][e2]), sc[1][e2 + 1]);
      }
      x = fmaxf(fmaxf(x, sc[0][15]), sc[1][15]);
      return max_pair32(fmaxf(x, y));
    };

    float l_run = 0.f;   // this lane's partial row sum (its 32 keys per step)
    const bf16x2 ones{(__bf16)1.0f, (__bf16)1.0f};
    f32x16 oacc[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t) oacc[t] = f32x16{};
    f32x16 mneg;   // -m in every element: the start of each S accumulator
    float mx = 0.f;   // row maximum of the current S (relative to the base)

    // K operand of QK MFMA i (k-step i / 2 over D, 32-key half i % 2) of the
    // stage at kb; V operand of PV MFMA i (16-key slice i / DT, output tile
    // i % DT) of the stage at vb.
    auto rdk = [&](int kb, int i) __attribute__((always_inline)) -> bf16x8 {
      return rd16(kb + (i & 1) * 32 * RB + (i >> 1) * 512);
    };
    auto rdv = [&](int vb, int i) __attribute__((always_inline)) -> bf16x8 {
      const int o = vb + (i / DT) * BLK + (i % DT) * 1024;
      const u32x2 lo = rdtr(v_off0 + o), hi = rdtr(v_off1 + o);
      return __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
    };
    // S^T = K Q^T of a step (no other work), accumulators from zero.
    auto qk_alone = [&](int kb, f32x16 (&sc)[2]) __attribute__((always_inline)) {
      constexpr int N = 2 * KS;
      bf16x8 kf[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) kf[i] = rdk(kb, i);
#pragma unroll
      for (int i = 0; i < N; ++i) {
        sc[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i % 3], qf[i >> 1], i < 2 ? f32x16{} : sc[i & 1], 0, 0, 0);
        if (i + 3 < N) kf[i % 3] = rdk(kb, i + 3);
      }
    };
    // Probabilities of element pair i (of 16) of S: 2^(s - m) for two keys,
    // packed to bf16.
    auto prob_pair = [&](const f32x16 (&sc)[2], int i) __attribute__((always_inline)) -> uint32_t {
      const int kk = i >> 2, jj = i & 3, h = kk >> 1, e = (kk & 1) * 8 + 2 * jj;
      return pack_bf16x2(__builtin_amdgcn_exp2f(sc[h][e]), __builtin_amdgcn_exp2f(sc[h][e + 1]));
    };
    // ls += the two probabilities of a packed pair (the row sum uses the
    // rounded probabilities the PV product uses)
    auto sum_pair = [&](uint32_t w, float& ls) __attribute__((always_inline)) {
      ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, ls, false);
    };
    auto pack_pb = [&](const uint32_t (&w)[16], bf16x8 (&pb)[4]) __attribute__((always_inline)) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) pb[kk] = __builtin_bit_cast(bf16x8, u32x4{w[4 * kk], w[4 * kk + 1], w[4 * kk + 2], w[4 * kk + 3]});
    };
    // Where a step's copies go: the first half after MFMAs ke, ke + E, .. of
    // phase A (ke: the groups before the wave's copy work), the second half
    // after MFMAs 0, E, 2E, .. of phase B; a step without phase A (an entry's
    // last) puts all of them in phase B.
    // In the fused kernel waves 4-7 do their copy work after KS groups of
    // phase A, waves 0-3 (and every wave of the other kernels) after kEarly:
    // the two waves of a SIMD (w and w + 4) then take the CU's one scalar unit
    // at different times, each while the other issues MFMAs. (The fused
    // kernel's copy work is twice as long; for the others this measured
    // slightly slower.)
    constexpr int HALF_C = LPW / 2;
    constexpr int kEarly = 2;   // phase A groups issued before a step's copy work
    constexpr int kLate = KS;   // (fused kernel, waves 4-7)
    auto copies_a = [&](int i, int ke) __attribute__((always_inline)) {
      if (ke == kEarly) {
        constexpr int E = 2 * KS / HALF_C;
        if (i % E == kEarly) copy_part(i / E);
      } else {
        constexpr int E = (2 * KS - kLate) / HALF_C;
        if (i >= kLate && (i - kLate) % E == 0) copy_part((i - kLate) / E);
      }
    };
    auto copies_b = [&](int i, bool all) __attribute__((always_inline)) {
      constexpr int E = 4 * DT / HALF_C, EA = 4 * DT / LPW;
      if (all) {
        if (i % EA == 0) copy_part(i / EA);
      } else if (i % E == 0) {
        copy_part(HALF_C + i / E);
      }
    };
    // Phase A of a step: S(j+1) = K Q^T from the stage at kb (accumulators
    // from -m) interleaved with the probabilities of S(j) (sc -> pb). Each
    // group is one MFMA, the operand read three MFMAs ahead and one element
    // pair of the softmax, fenced by a scheduling barrier so that the groups
    // keep this order (the compiler would otherwise gather the vector work
    // after the last MFMA and reorder the MFMAs, collapsing the read-ahead);
    // an empty use pins each pair in its group.
    // The first three K operands (kf, read by the caller before the step's
    // scalar work so that their latency overlaps it) and, in the last three
    // groups, the first three V operands of phase B (vf).
    // Groups [i0, i1) of phase A (a step issues the first groups before its
    // scalar copy work, so that the matrix pipe has work meanwhile); pack
    // ends the phase.
    auto phase_a = [&](int kb, int vb, bf16x8 (&kf)[3], bf16x8 (&vf)[3], const f32x16 (&sc)[2], f32x16 (&sn)[2],
                       uint32_t (&w)[16], bf16x8 (&pb)[4], int i0, int i1, int ke, bool pack) __attribute__((always_inline)) {
      constexpr int N = 2 * KS;
      constexpr int PER = 16 / N;   // element pairs per MFMA (1 for D = 128, 2 for D = 64)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = i0; i < i1; ++i) {
        sn[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i % 3], qf[i >> 1], i < 2 ? mneg : sn[i & 1], 0, 0, 0);
        if (i + 3 < N) kf[i % 3] = rdk(kb, i + 3);
        else vf[i + 3 - N] = rdv(vb, i + 3 - N);
        copies_a(i, ke);
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          w[i * PER + u] = prob_pair(sc, i * PER + u);
          asm volatile("" :: "v"(w[i * PER + u]));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if (pack) pack_pb(w, pb);
    };
    // The last step of an entry (no next scores): O^T += V^T P^T with the
    // probabilities of 16-key slice kk + 1 formed while the PV MFMAs of slice
    // kk run (slice 0 first, alone); all of the step's copies go here.
    auto phase_last = [&](int vb, const f32x16 (&sc)[2]) __attribute__((always_inline)) {
      constexpr int N = 4 * DT;
      constexpr int PER = 4 / DT;   // element pairs per MFMA (1 for D = 128, 2 for D = 64)
      uint32_t w[16];
      float ls[2] = {0.f, 0.f};
      bf16x8 vf[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) vf[i] = rdv(vb, i);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w[i] = prob_pair(sc, i);
        sum_pair(w[i], ls[i & 1]);
      }
      bf16x8 pk = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int kk = i / DT;
        oacc[i % DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i % 3], pk, oacc[i % DT], 0, 0, 0);
        if (i + 3 < N) vf[i % 3] = rdv(vb, i + 3);
        copies_b(i, true);
        if (kk + 1 < 4) {
#pragma unroll
          for (int u = 0; u < PER; ++u) {
            const int q = (kk + 1) * 4 + (i % DT) * PER + u;
            w[q] = prob_pair(sc, q);
            sum_pair(w[q], ls[q & 1]);
            asm volatile("" :: "v"(w[q]));
          }
        } else {
          asm volatile("" :: "v"(vf[(i + 1) % 3]));
        }
        if (i % DT == DT - 1 && kk + 1 < 4)
          pk = __builtin_bit_cast(bf16x8, u32x4{w[4 * kk + 4], w[4 * kk + 5], w[4 * kk + 6], w[4 * kk + 7]});
        __builtin_amdgcn_sched_barrier(0);
      }
      l_run += ls[0] + ls[1];
    };
    // Phase B of a step: O^T += V^T P^T from the stage at vb (operand reads
    // three ahead), in groups like phase A's: the row sums of P in the first
    // half of the groups, the row maximum of the next scores sn (already
    // masked) in the second half, when the last MFMAs of phase A, which wrote
    // sn, have long completed; returns the maximum relative to the base.
    // (vf: the first three V operands, read in phase A)
    auto phase_b = [&](int vb, bf16x8 (&vf)[3], const bf16x8 (&pb)[4], const f32x16 (&sn)[2])
        __attribute__((always_inline)) -> float {
      constexpr int N = 4 * DT;
      constexpr int PER = 32 / N;   // sums (first half) or max3 operations (second half) per MFMA
      float x[2] = {-INFINITY, -INFINITY};
      float ls[2] = {0.f, 0.f};
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < N; ++i) {
        oacc[i % DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i % 3], pb[i / DT], oacc[i % DT], 0, 0, 0);
        if (i + 3 < N) vf[i % 3] = rdv(vb, i + 3);
        copies_b(i, false);
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          if (i < N / 2) {
            const int q = i * PER + u;
            sum_pair(__builtin_bit_cast(u32x4, pb[q >> 2])[q & 3], ls[q & 1]);
            asm volatile("" :: "v"(ls[q & 1]));
          } else {
            const int q = (i - N / 2) * PER + u, h = q & 1, e = (q >> 1) * 2;
            x[h] = fmaxf(fmaxf(x[h], sn[h][e]), sn[h][e + 1]);
            asm volatile("" :: "v"(x[h]));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      l_run += ls[0] + ls[1];
      return max_pair32(fmaxf(x[0], x[1]));
    };
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
    auto kbase = [&](int pp) { return k_off + (pp & (kStages - 1)) * KTILE; };
    auto vbase = [&](int pp) { return (pp & (kStages - 1)) * VTILE; };

    // ---- S(0) with the exact row maximum as base
    f32x16 sa[2], sb[2];
    qk_alone(kbase(p), sa);
    if (n_full == 0) mask(sa, kbeg * kKv);
    {
      // Finite when the run's first step has a visible key for this row (always
      // so for the first run: key 0 is visible to every row). A row that sees no
      // key of the run's first step sees none of its later steps either (they
      // hold higher keys), so any base serves it.
      float m0 = rowmax(sa);
      if (m0 == -INFINITY) m0 = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) sa[h] -= m0;
#pragma unroll
      for (int e2 = 0; e2 < 16; ++e2) mneg[e2] = -m0;
    }

    const int last = nsteps - 1;
    // Two steps before its last one, an entry brings the next entry's queries
    // into L2 (one 128-byte line per lane), so that their load at the last
    // step does not wait for HBM. (Entries of one or two steps skip it.)
    const int touch_at = last - 2;
    auto touch_q = [&]() __attribute__((always_inline)) {
      touch_line(reinterpret_cast<const uint8_t*>(q_next) + half * 128, own_area);
    };
    // FUSED: the keys of this entry's query rows are new keys of this call.
    // Where this wave's block of step jj (ring position p) holds some of them
    // (an entry's last steps), the wave writes those rows from the stage into
    // the block's place in its cache (the destination recorded when the block
    // was copied; -1 where the call writes nothing). A block the entry owns
    // whole is written by LPW stores issued after the step's last copy
    // (write_late): the step's barrier then leaves them in flight and the next
    // step's barrier completes them. A block owned in part (a request's last
    // rows, or tiles of fewer than 16 positions) is written at the step's
    // start, before its copies (write_early).
    constexpr int NST = LPW;        // store instructions per block
    // the first step (from kbeg) that holds a key of the entry's own rows: the
    // steps before it write nothing
    const int own_j0 = (P + row0) / kKv - kbeg;
    auto own_span = [&](int jj, int& key0, int& lo, int& hi) __attribute__((always_inline)) -> int {
      key0 = ((kbeg + jj) * (kKv / kBs) + bs) * kBs;
      lo = max(key0, P + row0);
      hi = min(key0 + kBs, P + row0 + nvalid);
      return __builtin_amdgcn_readlane(dring, p & (kStages - 1));
    };
    // The block as staged: lane l's 16 bytes at 1024 it + 16 l of its slot
    // are the bytes it copied, chunk 4 it + l / 16 of key ckey, so they go to
    // the same offset in the destination block as they came from (off_c).
    auto own_chunk = [&](int it) __attribute__((always_inline)) -> u32x4 {
      const uint32_t sb = slot0 - lds0 + uint32_t(p & (kStages - 1)) * stage_stride;
      return *reinterpret_cast<const u32x4*>(lds + sb + it * 1024 + lane * 16);
    };
    auto own_dst = [&](int dstb) __attribute__((always_inline)) -> uint8_t* {
      return reinterpret_cast<uint8_t*>(is_v ? a.vw : a.kw) + uint64_t(uint32_t(dstb)) * blk_bytes +
             uint32_t(g) * (kBs * RB) + off_c;
    };
    auto write_early = [&](int jj) __attribute__((always_inline)) {
      int key0, lo, hi;
      const int dstb = own_span(jj, key0, lo, hi);
      if (uint32_t(dstb) >= uint32_t(a.num_blocks) || lo >= hi || (lo == key0 && hi == key0 + kBs)) return;
      u32x4 t[LPW];
#pragma unroll
      for (int it = 0; it < LPW; ++it) t[it] = own_chunk(it);
      uint8_t* dp = own_dst(dstb);
      const bool mine = key0 + ckey >= lo && key0 + ckey < hi;
#pragma unroll
      for (int it = 0; it < LPW; ++it)
        if (mine) *reinterpret_cast<u32x4*>(dp + 64 * it) = t[it];
    };
    auto write_late = [&](int jj) __attribute__((always_inline)) -> bool {
      int key0, lo, hi;
      const int dstb = own_span(jj, key0, lo, hi);
      if (uint32_t(dstb) >= uint32_t(a.num_blocks) || lo != key0 || hi != key0 + kBs) return false;
      u32x4 t[LPW];
#pragma unroll
      for (int it = 0; it < LPW; ++it) t[it] = own_chunk(it);
      uint8_t* dp = own_dst(dstb);
#pragma unroll
      for (int it = 0; it < LPW; ++it) {
        // (a store of more than 8 bytes reads its data registers after issue:
        // wait states before an instruction may write them)
        asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 1" :: "v"(dp + 64 * it), "v"(t[it]) : "memory");
      }
      return true;
    };
    // The step barrier after write_late's stores: they stay in flight with
    // the step's copies.
    auto step_barrier_w = [&](bool keep, bool late) __attribute__((always_inline)) {
      if (keep && late) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(LPW + NST));
      else if (keep) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(LPW));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    };
    // Step j < nsteps - 1 at ring position p: current S in sc, next S into sn.
    auto step = [&](int j, f32x16 (&sc)[2], f32x16 (&sn)[2]) __attribute__((always_inline)) {
      if constexpr (FUSED) {
        if (j >= own_j0) write_early(j);
      }
      bf16x8 kf[3], vf[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) kf[i] = rdk(kbase(p + 1), i);
      if (j == touch_at) touch_q();
      rebase(sc);
      bf16x8 pb[4];
      uint32_t w[16];
      bool direct;
      if (!FUSED || wave < 4) {
        phase_a(kbase(p + 1), vbase(p), kf, vf, sc, sn, w, pb, 0, kEarly, kEarly, false);
        direct = issue(p + kAhead, true);
        phase_a(kbase(p + 1), vbase(p), kf, vf, sc, sn, w, pb, kEarly, 2 * KS, kEarly, true);
      } else {
        phase_a(kbase(p + 1), vbase(p), kf, vf, sc, sn, w, pb, 0, kLate, kLate, false);
        direct = issue(p + kAhead, true);
        phase_a(kbase(p + 1), vbase(p), kf, vf, sc, sn, w, pb, kLate, 2 * KS, kLate, true);
      }
      if (j + 1 >= n_full) mask(sn, (kbeg + j + 1) * kKv);
      mx = phase_b(vbase(p), vf, pb, sn);
      if (FUSED && j >= own_j0) step_barrier_w(direct, write_late(j));
      else step_barrier(direct);
      ++p;
    };
    int j = 0;
    // two steps per iteration so the S buffers alternate without copies
    for (; j + 1 < last; j += 2) {
      step(j, sa, sb);
      step(j + 1, sb, sa);
    }
    if (j < last) {
      step(j, sa, sb);
#pragma unroll
      for (int h = 0; h < 2; ++h) sa[h] = sb[h];
      ++j;
    }
    {   // the entry's last step: P and PV only. qf is no longer needed: the
        // next entry's Q is loaded now, ahead of this step's table word and
        // copies, so that this step's barrier completes it.
      if constexpr (FUSED) {
        if (last >= own_j0) write_early(last);
      }
      load_q(q_next);
      load_desc(e + grid);
      const bool direct = issue(p + kAhead, true);
      rebase(sa);
      phase_last(vbase(p), sa);
      if (FUSED && last >= own_j0) step_barrier_w(direct, write_late(last));
      else step_barrier(direct);
      ++p;
    }

    const float l_tot = sum_pair32(l_run);
    if constexpr (SPLIT) {
      if (!row_ok) continue;
      const int64_t prow = int64_t(split) * a.part_rows + qrow * a.hq + head;
      float* po = a.part_o + prow * D;
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
      if (half == 0) a.part_lse[prow] = any ? -mneg[0] + __log2f(l_tot) : -INFINITY;
    } else {
      // The output goes through this wave's staging area: a lane holds 4
      // consecutive d of its row per (t, gq), so direct stores would write 32
      // rows in 8-byte pieces per instruction. Each round stages a range of d
      // (HD values) of all 32 rows and reads it back as rows of 16-byte
      // chunks, so that each store covers whole 128-byte lines of HD values
      // (16-byte chunk c of staged row r at position c ^ (r % CPR):
      // conflict-free writes and reads). Lanes read what other lanes wrote:
      // the hardware keeps a wave's LDS accesses in order, and empty asm
      // statements with a memory clobber keep the compiler from reusing, for
      // a lane, values it loaded before another lane's writes (as it may, for
      // memory it sees no other thread write).
      constexpr int HD = G::STAGING / (32 * 2);   // d values per round (64)
      constexpr int CPR = HD / 8;                // 16-byte chunks per staged row
      constexpr int TPR = HD / 32;               // output tiles per round
      constexpr int RPI = 64 / CPR;              // staged rows per read instruction
      static_assert(D % HD == 0 && CPR == 8, "staging rounds");
      const float inv = row_ok ? __builtin_amdgcn_rcpf(l_tot) : 0.f;
      uint8_t* stg = lds + G::RING + wave * G::STAGING;
      // Opaque copies of the values the addresses below derive from: without
      // them the compiler computes those (entry- or lane-invariant) addresses
      // before the steps and keeps them live across the step loop.
      int ln = lane, q0 = qrow0, nv = nvalid, hg = g * a.group;
      asm volatile("" : "+v"(ln), "+s"(q0), "+s"(nv), "+s"(hg));
      const int l32e = ln & 31, halfe = ln >> 5;
#pragma unroll
      for (int rd = 0; rd < D / HD; ++rd) {
#pragma unroll
        for (int tt = 0; tt < TPR; ++tt)
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            const int t = rd * TPR + tt, c = tt * 4 + gq;   // d = 32 t + 8 gq + 4 half ..
            const u32x2 w{pack_bf16x2(oacc[t][gq * 4 + 0] * inv, oacc[t][gq * 4 + 1] * inv),
                          pack_bf16x2(oacc[t][gq * 4 + 2] * inv, oacc[t][gq * 4 + 3] * inv)};
            *reinterpret_cast<u32x2*>(stg + l32e * (HD * 2) + ((c ^ (l32e % CPR)) << 4) + halfe * 8) = w;
          }
        asm volatile("" ::: "memory");
        // all of the round's reads first, then the stores of the rows that exist
        u32x4 v[32 / RPI];
#pragma unroll
        for (int q = 0; q < 32 / RPI; ++q) {
          const int r = q * RPI + ln / CPR, c = ln % CPR;
          v[q] = *reinterpret_cast<const u32x4*>(stg + r * (HD * 2) + ((c ^ (r % CPR)) << 4));
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int q = 0; q < 32 / RPI; ++q) {
          const int r = q * RPI + ln / CPR, c = ln % CPR;
          // the staged row's column of the tile, its head and position
          const uint32_t mr = uint32_t(wave * 32 + r);
          const int hr = int((mr * tdiv) >> 16);
          const int pr = int(mr) - hr * a.per_tile;
          if (hr < a.group && pr < nv)
            *reinterpret_cast<u32x4*>(a.out + ((int64_t(q0) + pr) * a.hq + hg + hr) * D + rd * HD + c * 8) = v[q];
        }
      }
    }
  }
  // Every copy the cursor issued was consumed: the cursor runs out with the
  // last entry, and every issued step is computed before the loop ends.
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
                     static_cast<u32x4*>(v_cache), block_table, bt_stride, cu_suffix_dev,
                     prefix_len_dev, batch, num_kv_heads, head_dim, num_blocks);
  return check_launch("kv_append launch");
}

namespace {

// Checks shared by the attention entry points; fills the launch arguments.
struct AttnLaunch {
  AttnArgs args;
  int32_t grid = 0, splits = 1;
  int64_t rows = 0;
};
cw_status check_attn(const char* what, const void* q, const void* k_cache, const void* v_cache,
                     const int32_t* block_table, int32_t bt_stride, const int32_t* cu_suffix_dev,
                     const int32_t* prefix_len_dev, const int32_t* cu_suffix_host,
                     const int32_t* prefix_len_host, int32_t batch, int32_t num_q_heads,
                     int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t num_blocks,
                     float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev, const void* out,
                     AttnLaunch* L, const int32_t* append_bt_host = nullptr) {
  const std::string w(what);
  // the fused call reads no device block table or offsets: its plan carries them
  const bool fused = append_bt_host != nullptr;
  if (!q || !k_cache || !v_cache || !out || (!fused && (!block_table || !cu_suffix_dev || !prefix_len_dev)))
    return cw::fail(CW_EINVAL, w + ": a required pointer is NULL");
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0)
    return cw::fail(CW_EINVAL, w + ": num_q_heads must be a positive multiple of num_kv_heads");
  if (num_blocks < 1) return cw::fail(CW_EINVAL, w + ": num_blocks must be >= 1");
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    return cw::fail(CW_EINVAL, w + ": softmax_scale must be finite and positive");
  if (head_dim != 64 && head_dim != 128) return cw::fail(CW_EUNSUPPORTED, w + ": head_dim must be 64 or 128");
  if (block_size != kBs) return cw::fail(CW_EUNSUPPORTED, w + ": block_size must be 16");
  const int group = num_q_heads / num_kv_heads;
  if (group > cw::kMaxGroup) return cw::fail(CW_EUNSUPPORTED, w + ": more than 128 query heads per KV head");
  if (num_kv_heads > cw::kMaxKvHeads) return cw::fail(CW_EUNSUPPORTED, w + ": more than 65536 KV heads");
  cw_status st = cw::check_batch(cu_suffix_host, prefix_len_host, batch, block_size, bt_stride, &L->rows);
  if (st != CW_OK) return st;
  AttnArgs& a = L->args;
  st = cw::check_plan_header(what, plan_host, cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads,
                             head_dim, &L->grid, &L->splits, &a.fp_lo, &a.fp_hi, &a.num_entries, append_bt_host,
                             bt_stride, num_blocks);
  if (st != CW_OK) return st;
  if (L->grid > 0 && !plan_dev) return cw::fail(CW_EINVAL, w + ": plan_dev is required");
  a.q = static_cast<const uint16_t*>(q);
  a.kc = static_cast<const uint16_t*>(k_cache);
  a.vc = static_cast<const uint16_t*>(v_cache);
  a.bt = fused ? plan_dev + plan_host[cw::kHdrTable] : block_table;
  a.kn = nullptr;
  a.vn = nullptr;
  a.kw = nullptr;
  a.vw = nullptr;
  a.total_rows = 0;
  a.plan = plan_dev;
  a.out = static_cast<uint16_t*>(const_cast<void*>(out));
  a.part_o = nullptr;
  a.part_lse = nullptr;
  a.part_rows = L->rows * num_q_heads;
  a.bt_stride = bt_stride;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.group = group;
  a.per_tile = cw::tile_positions(group);
  a.num_blocks = num_blocks;
  a.c_log2 = softmax_scale * 1.4426950408889634f;
  return CW_OK;
}

template <bool SPLIT, bool FUSED = false>
void launch_attn(int head_dim, const AttnLaunch& L, hipStream_t s) {
  if (head_dim == 128)
    hipLaunchKernelGGL((suffix_prefill_attn_kernel<128, SPLIT, FUSED>), dim3(unsigned(L.grid)), dim3(kAttnThreads),
                       0, s, L.args);
  else
    hipLaunchKernelGGL((suffix_prefill_attn_kernel<64, SPLIT, FUSED>), dim3(unsigned(L.grid)), dim3(kAttnThreads),
                       0, s, L.args);
}

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
                                            float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev,
                                            void* out, void* stream) {
  AttnLaunch L;
  cw_status st = check_attn("suffix_prefill_attn", q, k_cache, v_cache, block_table, bt_stride, cu_suffix_dev,
                            prefix_len_dev, cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads,
                            head_dim, block_size, num_blocks, softmax_scale, plan_host, plan_dev, out, &L);
  if (st != CW_OK) return st;
  if (L.splits != 1)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn: the plan has splits; use cw_suffix_prefill_attn_split");
  if (L.rows == 0 || L.grid == 0) return cw::ok();
  launch_attn<false>(head_dim, L, static_cast<hipStream_t>(stream));
  return check_launch("suffix_prefill_attn launch");
}

extern "C" cw_status cw_suffix_prefill_append_attn(const void* q, const void* k_new, const void* v_new,
                                                   void* k_cache, void* v_cache, const int32_t* block_table_host,
                                                   int32_t bt_stride, const int32_t* cu_suffix_host,
                                                   const int32_t* prefix_len_host, int32_t batch,
                                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                                   int32_t block_size, int32_t num_blocks, float softmax_scale,
                                                   const int32_t* plan_host, const int32_t* plan_dev, void* out,
                                                   void* stream) {
  if (!k_new || !v_new || !block_table_host)
    return cw::fail(CW_EINVAL, "suffix_prefill_append_attn: a required pointer is NULL");
  AttnLaunch L;
  cw_status st = check_attn("suffix_prefill_append_attn", q, k_cache, v_cache, nullptr, bt_stride, nullptr, nullptr,
                            cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, head_dim, block_size,
                            num_blocks, softmax_scale, plan_host, plan_dev, out, &L, block_table_host);
  if (st != CW_OK) return st;
  if (L.rows == 0 || L.grid == 0) return cw::ok();
  if (num_blocks > cw::kMaxAppendBlocks)
    return cw::fail(CW_EUNSUPPORTED, "suffix_prefill_append_attn: num_blocks must be below 2^27");
  L.args.total_rows = int32_t(L.rows);
  L.args.kn = static_cast<const uint16_t*>(k_new);
  L.args.vn = static_cast<const uint16_t*>(v_new);
  L.args.kw = static_cast<uint16_t*>(k_cache);
  L.args.vw = static_cast<uint16_t*>(v_cache);
  launch_attn<false, true>(head_dim, L, static_cast<hipStream_t>(stream));
  return check_launch("suffix_prefill_append_attn launch");
}

extern "C" int64_t cw_suffix_prefill_split_workspace_bytes(int64_t total_rows, int32_t num_q_heads,
                                                           int32_t head_dim, int32_t num_splits) {
  if (total_rows < 0 || num_q_heads < 1 || (head_dim != 64 && head_dim != 128) || num_splits < 1 ||
      num_splits > cw::kMaxSplits)
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
                                                  float softmax_scale, const int32_t* plan_host,
                                                  const int32_t* plan_dev, void* workspace, int64_t workspace_bytes,
                                                  void* out, void* stream) {
  AttnLaunch L;
  cw_status st = check_attn("suffix_prefill_attn_split", q, k_cache, v_cache, block_table, bt_stride,
                            cu_suffix_dev, prefix_len_dev, cu_suffix_host, prefix_len_host, batch, num_q_heads,
                            num_kv_heads, head_dim, block_size, num_blocks, softmax_scale, plan_host, plan_dev,
                            out, &L);
  if (st != CW_OK) return st;
  const int64_t need = cw_suffix_prefill_split_workspace_bytes(L.rows, num_q_heads, head_dim, L.splits);
  if (!workspace || workspace_bytes < need)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn_split: workspace must hold " + std::to_string(need) + " bytes");
  if (L.rows == 0 || L.grid == 0) return cw::ok();
  auto* s = static_cast<hipStream_t>(stream);
  L.args.part_o = static_cast<float*>(workspace);
  L.args.part_lse = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                             split_lse_offset(L.args.part_rows, head_dim, L.splits));
  launch_attn<true>(head_dim, L, s);
  st = check_launch("suffix_prefill_attn_split launch");
  if (st != CW_OK) return st;
  return launch_merge(L.args.part_o, L.args.part_lse, L.splits, L.args.part_rows, head_dim, out, s);
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

// ---------------------------------------------------------------------------
// Split attention without allocation. The split path's partial results (fp32
// O per run and row, and the per-row log-sum-exp) go to a file-scope device
// array instead of a caller workspace, for callers that cannot allocate. Each
// GPU the library runs on holds its own copy of the array for the life of the
// process. The host takes the array's device address once per device (with
// that device current) through hipGetSymbolAddress and passes that address to
// the kernels; the array's name itself is never used as a device pointer on
// the host.
// ---------------------------------------------------------------------------
namespace {

constexpr int64_t kScratchBytes = cw::kNoAllocScratchBytes;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (taken on first use).
cw_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return cw::fail(CW_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return cw::fail(CW_EUNSUPPORTED, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return cw::fail(CW_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CW_OK;
}

}  // namespace

extern "C" int64_t cw_noalloc_scratch_bytes(void) { return kScratchBytes; }

extern "C" cw_status cw_suffix_prefill_attn_split_noalloc(
    const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table, int32_t bt_stride,
    const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev, const int32_t* cu_suffix_host,
    const int32_t* prefix_len_host, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
    int32_t block_size, int32_t num_blocks, float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev,
    void* out, void* stream) {
  AttnLaunch L;
  cw_status st = check_attn("suffix_prefill_attn_split_noalloc", q, k_cache, v_cache, block_table, bt_stride,
                            cu_suffix_dev, prefix_len_dev, cu_suffix_host, prefix_len_host, batch, num_q_heads,
                            num_kv_heads, head_dim, block_size, num_blocks, softmax_scale, plan_host, plan_dev,
                            out, &L);
  if (st != CW_OK) return st;
  const int64_t need = cw_suffix_prefill_split_workspace_bytes(L.rows, num_q_heads, head_dim, L.splits);
  if (need > kScratchBytes)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn_split_noalloc: the batch needs " + std::to_string(need) +
                                   " bytes of partial results; the built-in scratch holds " +
                                   std::to_string(kScratchBytes));
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != CW_OK) return st;
  if (L.rows == 0 || L.grid == 0) return cw::ok();
  auto* s = static_cast<hipStream_t>(stream);
  // Every part of every row is written by the split kernel (empty runs write
  // zeros and -inf) before the merge reads it, so nothing needs clearing.
  L.args.part_o = static_cast<float*>(ws);
  L.args.part_lse = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) +
                                             split_lse_offset(L.args.part_rows, head_dim, L.splits));
  launch_attn<true>(head_dim, L, s);
  st = check_launch("suffix_prefill_attn_split_noalloc launch");
  if (st != CW_OK) return st;
  return launch_merge(L.args.part_o, L.args.part_lse, L.splits, L.args.part_rows, head_dim, out, s);
}

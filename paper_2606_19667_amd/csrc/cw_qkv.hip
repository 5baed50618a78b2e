// Device half of libcw for gfx950 (MI355X): the suffix QKV projection with
// rotary embedding, fused with the KV append.
//
// Paper Sec. 1 and 2.1: a prefix hit removes every per-layer prefill step of
// the cached tokens; for the suffix tokens the layer still projects each
// hidden state to its query, key and value heads, rotates queries and keys by
// their absolute position, and stores the new keys and values in the
// request's cache blocks. This kernel does those three steps in one pass:
//
//   y = x W^T (+ b)          x [T, hidden], W [(Hq + 2 Hkv) D, hidden]
//   q, k = rope(y_q, y_k)    rotate-half form at position P_r + i
//   q -> q_out [T, Hq, D];  k -> K cache [blk][g][slot][d];
//   v -> V cache [blk][g][slot][d]
//
// Design (one workgroup = 8 wavefronts = one 256-feature x 256-token tile):
//  * The product is formed as C^T = W x^T with v_mfma_f32_16x16x32_bf16:
//    A = 16 rows of W, B = 16 token rows of x, 32 hidden per instruction. In
//    the 16x16 accumulator a lane holds one token and 4 consecutive features,
//    so everything the epilogue needs per element (position, block, slot) is
//    per lane. This shape sustains a higher rate than 32x32x16 on random data
//    (the card's power limit lowers the clock less for it).
//  * Wave (wf, wt) owns features {j0 .. j0 + 31} and {j0 + D/2 .. + 31} of one
//    head (four 16-row blocks) and 128 tokens (eight 16-token blocks). The
//    blocks j0 + 16 p and j0 + D/2 + 16 p are exactly rotary pairs
//    (j, j + D/2), which therefore sit in the same lane and register of two
//    accumulators: the rotation needs no data exchange.
//  * Hidden is walked in steps of 64 (two MFMA k-steps). Two LDS stages of
//    64 KB (256 W rows then 256 x rows, 128 bytes each) are filled by
//    LDS-direct loads (global_load_lds, no registers) one step ahead of their
//    use; one barrier per step. Each load instruction brings 8 whole 128-byte
//    rows (copies of whole lines out of L2 run at several times the rate of
//    half-line copies). The 16-byte chunk c of LDS row r holds global chunk
//    c ^ ((r >> 1) & 7), so the 16 rows read by one operand load hit distinct
//    banks. An odd count of 32 hidden ends with a half step whose upper
//    chunks are not used.
//  * Within a step a wave loads the first k-step's operands, then issues its
//    products in groups of one token block, each group followed by operand
//    loads of the second k-step and one of the next step's copies; then the
//    second k-step's products. The copies are inline asm, which the compiler
//    does not track: tracked LDS-direct loads make it wait for every LDS read
//    before the first product.
//  * Tiles are numbered XCD-major (workgroup b runs on XCD b % 8), and within
//    an XCD feature tiles vary fastest in groups of 8, so the workgroups that
//    run together on one L2 share their W and x rows.
//  * fp32 accumulation; bias, rotation (fp32 cos/sin from a table the host
//    computes in fp64) and one bf16 rounding in the epilogue.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>

#include "cw_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 512;                  // 8 wavefronts
constexpr int kTileF = 256;                    // output features per workgroup
constexpr int kTileT = 256;                    // tokens per workgroup
constexpr int kStep = 64;                      // hidden elements per pipeline step
constexpr int kRow = kStep * 2;                // bytes of one staged row (one 128-byte line)
constexpr int kPartW = kTileF * kRow;          // 32 KB: the W rows of a stage
constexpr int kStage = kPartW + kTileT * kRow; // + 32 KB of x rows
constexpr int kStages = 2;
constexpr int kAhead = kStages - 1;            // steps in flight (the loop's waits assume one)
constexpr int kCopiesW = kPartW / 1024 / 8;    // 1 KB LDS-direct copies per wave and step: W rows
constexpr int kCopiesX = kTileT * kRow / 1024 / 8;   // and x rows
constexpr int kCopies = kCopiesW + kCopiesX;
constexpr int kGroupF = 8;                     // feature tiles per XCD group
constexpr int kBs = cw::kBlockSize;
static_assert(kCopiesW == 4 && kCopiesX == 4, "8 rows per copy, 32 W and 32 x rows per wave");
static_assert(kStages * kStage <= 160 * 1024, "LDS of one CU");
static_assert(kAhead == 1, "each step waits for all of its copies");

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// One load-to-LDS copy: lane l's 16 bytes at src land at dst + 16 l (dst
// wave-uniform, through M0). The compiler does not count it: the kernel's own
// waits complete it.
__device__ __forceinline__ void copy16_to_lds(const void* src, lds_void_t* dst) {
  const uint32_t m = __builtin_amdgcn_readfirstlane(uint32_t(reinterpret_cast<uintptr_t>(dst)));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" :: "v"(src), "s"(m) : "memory");
}

// s_waitcnt immediates (gfx9 encoding): vmcnt(n) with lgkmcnt(0), expcnt untouched.
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 15) | (7 << 4) | ((n >> 4) << 14); }

// Chunk swizzle of staged row r (128-byte rows, eight 16-byte chunks): the
// 16 rows of an operand load, two per 256 bytes of banks, take 8 distinct
// positions per row parity.
__device__ __forceinline__ int row_swz(int r) { return (r >> 1) & 7; }

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void qkv_rope_append_kernel(const uint8_t* __restrict__ x, const uint8_t* __restrict__ w,
                            const uint16_t* __restrict__ bias, const float* __restrict__ rope,
                            int T, int hidden, int n_feat, uint16_t* __restrict__ q_out,
                            uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
                            const int32_t* __restrict__ bt, int bt_stride, const int32_t* __restrict__ cu,
                            const int32_t* __restrict__ plen, int batch, int hq, int hkv, int num_blocks,
                            int n_ftiles, int n_ttiles, int per_xcd) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kStage];

  // ---- tile of this workgroup
  const int b = blockIdx.x;
  const int L = (b & 7) * per_xcd + (b >> 3);
  if (L >= n_ftiles * n_ttiles) return;
  const int grp = L / (kGroupF * n_ttiles);
  const int gf = min(kGroupF, n_ftiles - grp * kGroupF);
  const int rem = L - grp * kGroupF * n_ttiles;
  const int tt = rem / gf;
  const int ft = grp * kGroupF + rem % gf;
  const int f0 = ft * kTileF;
  const int t0 = tt * kTileT;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- staging role: W rows 32 wave .. + 31 and x rows 32 wave .. + 31 of
  // each step; copy i brings 8 rows, lane l chunk l % 8 of row l / 8 (LDS
  // position l % 8 holds global chunk (l % 8) ^ row_swz(row)).
  const int64_t hb = int64_t(hidden) * 2;   // bytes per row of W and x
  const uint8_t* src[kCopies];
  int chunk[kCopies];
#pragma unroll
  for (int i = 0; i < kCopies; ++i) {
    const int row = i < kCopiesW ? 32 * wave + 8 * i + (lane >> 3) : 32 * wave + 8 * (i - kCopiesW) + (lane >> 3);
    chunk[i] = (lane & 7) ^ row_swz(row);
    src[i] = i < kCopiesW ? w + int64_t(min(f0 + row, n_feat - 1)) * hb : x + int64_t(min(t0 + row, T - 1)) * hb;
  }
  const int nk = (hidden + kStep - 1) / kStep;
  const bool half_last = (hidden % kStep) != 0;   // the last step holds 32 hidden
  // copy i of a step into stage st
  auto issue_one = [&](int step, int st, int i) __attribute__((always_inline)) {
    uint8_t* dst = lds + st * kStage;
    // (past the row's end in a half step the lane copies the chunk 4 below,
    // which nothing reads)
    const bool cut = half_last && step == nk - 1;
    const int c = (cut && chunk[i] >= 4) ? chunk[i] - 4 : chunk[i];
    const int off = i < kCopiesW ? (32 * wave + 8 * i) * kRow : kPartW + (32 * wave + 8 * (i - kCopiesW)) * kRow;
    copy16_to_lds(src[i] + int64_t(step) * kRow + c * 16, (lds_void_t*)(dst + off));
  };
  auto issue = [&](int step, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kCopies; ++i) issue_one(step, st, i);
  };

  // ---- operand rows of this wave
  constexpr int kWavesPerHead = D / 64;
  const int wf = wave & 3, wt = wave >> 2;
  const int head_l = wf / kWavesPerHead;
  const int j0 = (wf % kWavesPerHead) * 32;
  const int arow0 = head_l * D + j0;
  const int brow = wt * 128;
  const int l16 = lane & 15;
  const int g4 = lane >> 4;
  // 16-row block starting at a multiple of 16 rows, k-step ks of the stage:
  // lane reads row l16, chunk 4 ks + g4 (swizzled)
  const int so0 = l16 * kRow + ((g4 ^ row_swz(l16)) << 4);
  const int so1 = l16 * kRow + (((4 + g4) ^ row_swz(l16)) << 4);
  // feature blocks: fa = 0, 1 -> j0 + 16 fa; fa = 2, 3 -> j0 + D/2 + 16 (fa - 2)
  int arow[4];
#pragma unroll
  for (int fa = 0; fa < 4; ++fa) arow[fa] = arow0 + (fa >> 1) * (D / 2) + (fa & 1) * 16;

  f32x4 acc[4][8];
#pragma unroll
  for (int fa = 0; fa < 4; ++fa)
#pragma unroll
    for (int tb = 0; tb < 8; ++tb) acc[fa][tb] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int s = 0; s < kAhead; ++s)
    if (s < nk) issue(s, s);

  for (int k = 0; k < nk; ++k) {
    // this step's copies have landed, in every wave; then the stage of step
    // k - 1 is free for step k + 1
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    // the next step's copies go out with the first k-step's products (in the
    // last step they copy that step's rows again into the free stage: the
    // loop's end waits for them)
    const int nxt = min(k + kAhead, nk - 1);

    // The first k-step's operands, then its products in groups of one token
    // block (4 MFMAs), each followed by loads of the second k-step's operands
    // into the registers the group has consumed; then the second k-step's
    // products. Scheduling barriers keep this order. A half step loads the
    // second k-step's operands too and skips its products.
    const uint8_t* st = lds + (k % kStages) * kStage;
    auto ld = [&](int row, int so) __attribute__((always_inline)) -> bf16x8 {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(st + row * kRow + so));
    };
    bf16x8 a0[4], a1[4], bx[8];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fa = 0; fa < 4; ++fa) a0[fa] = ld(arow[fa], so0);
#pragma unroll
    for (int tb = 0; tb < 8; ++tb) bx[tb] = ld(kTileF + brow + 16 * tb, so0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int tb = 0; tb < 8; ++tb) {
#pragma unroll
      for (int fa = 0; fa < 4; ++fa)
        acc[fa][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[fa], bx[tb], acc[fa][tb], 0, 0, 0);
      bx[tb] = ld(kTileF + brow + 16 * tb, so1);
      if (tb < 4) a1[tb] = ld(arow[tb], so1);
      issue_one(nxt, (k + kAhead) % kStages, tb);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (!(half_last && k == nk - 1)) {
#pragma unroll
      for (int tb = 0; tb < 8; ++tb) {
#pragma unroll
        for (int fa = 0; fa < 4; ++fa)
          acc[fa][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[fa], bx[tb], acc[fa][tb], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));

  // ---- epilogue: bias, rotation, bf16 rounding, stores
  const int hf = (f0 + head_l * D) / D;
  if (hf >= hq + 2 * hkv) return;
  const int kind = hf < hq ? 0 : (hf < hq + hkv ? 1 : 2);
  const int g = kind == 1 ? hf - hq : hf - hq - hkv;
  // element e of acc[fa][tb]: feature j0 + 16 (fa & 1) + 4 g4 + e (+ D/2 for fa >= 2), token brow + 16 tb + l16
  float bb[4][4];
#pragma unroll
  for (int fa = 0; fa < 4; ++fa) {
    if (bias) {
      const u32x2 v = *reinterpret_cast<const u32x2*>(bias + int64_t(hf) * D + j0 + (fa >> 1) * (D / 2) + (fa & 1) * 16 + 4 * g4);
      bb[fa][0] = bf16_lo(v[0]); bb[fa][1] = bf16_hi(v[0]); bb[fa][2] = bf16_lo(v[1]); bb[fa][3] = bf16_hi(v[1]);
    } else {
      bb[fa][0] = bb[fa][1] = bb[fa][2] = bb[fa][3] = 0.f;
    }
  }

#pragma unroll
  for (int tb = 0; tb < 8; ++tb) {
    const int t = t0 + brow + 16 * tb + l16;
    if (t >= T) continue;
    int lo = 0, hi = batch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= t) lo = mid;
      else hi = mid - 1;
    }
    const int pos = plen[lo] + (t - cu[lo]);
    int blk = 0, slot = 0;
    if (kind != 0) {
      blk = bt[int64_t(lo) * bt_stride + pos / kBs];
      if (blk < 0 || blk >= num_blocks) continue;
      slot = pos % kBs;
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int j = j0 + 16 * p + 4 * g4;   // rotary index of element 0
      float o0[4], o1[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o0[e] = acc[p][tb][e] + bb[p][e];
        o1[e] = acc[p + 2][tb][e] + bb[p + 2][e];
      }
      if (kind != 2) {
        const float* cs = rope + (int64_t(pos) * (D / 2) + j) * 2;
        const f32x4 c01 = *reinterpret_cast<const f32x4*>(cs);
        const f32x4 c23 = *reinterpret_cast<const f32x4*>(cs + 4);
        const float c[4] = {c01[0], c01[2], c23[0], c23[2]};
        const float sn[4] = {c01[1], c01[3], c23[1], c23[3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float av = o0[e], bv = o1[e];
          o0[e] = av * c[e] - bv * sn[e];
          o1[e] = bv * c[e] + av * sn[e];
        }
      }
      if (kind == 0) {
        uint16_t* qp = q_out + (int64_t(t) * hq + hf) * D + j;
        *reinterpret_cast<u32x2*>(qp) = u32x2{pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3])};
        *reinterpret_cast<u32x2*>(qp + D / 2) = u32x2{pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3])};
      } else {
        // k or v: row `slot` of the (block, head) in its cache, [blk][g][slot][d]
        uint16_t* cp = (kind == 1 ? k_cache : v_cache) + ((int64_t(blk) * hkv + g) * kBs + slot) * D + j;
        *reinterpret_cast<u32x2*>(cp) = u32x2{pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3])};
        *reinterpret_cast<u32x2*>(cp + D / 2) = u32x2{pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3])};
      }
    }
  }
}

cw_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return cw::fail(CW_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  return cw::ok();
}

}  // namespace

extern "C" cw_status cw_qkv_rope_append(const void* x, const void* w, const void* bias, const float* rope,
                                        int32_t rope_len, int32_t hidden, void* q_out, void* k_cache,
                                        void* v_cache, const int32_t* block_table, int32_t bt_stride,
                                        const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                        const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                        int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t block_size, int32_t num_blocks, void* stream) {
  const char* what = "qkv_rope_append";
  if (!w || !rope || !k_cache || !v_cache || !block_table || !cu_suffix_dev || !prefix_len_dev)
    return cw::fail(CW_EINVAL, std::string(what) + ": a required pointer is NULL");
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0)
    return cw::fail(CW_EINVAL, std::string(what) + ": num_q_heads must be a positive multiple of num_kv_heads");
  if (num_blocks < 1) return cw::fail(CW_EINVAL, std::string(what) + ": num_blocks must be >= 1");
  if (head_dim != 64 && head_dim != 128)
    return cw::fail(CW_EUNSUPPORTED, std::string(what) + ": head_dim must be 64 or 128");
  if (block_size != kBs) return cw::fail(CW_EUNSUPPORTED, std::string(what) + ": block_size must be 16");
  if (hidden < kStep / 2 || hidden % (kStep / 2) != 0 || hidden > (1 << 20))
    return cw::fail(CW_EUNSUPPORTED, std::string(what) + ": hidden must be a multiple of 32 in [32, 2^20]");
  if (rope_len < 0) return cw::fail(CW_EINVAL, std::string(what) + ": rope_len must be >= 0");
  int64_t rows = 0;
  cw_status st = cw::check_batch(cu_suffix_host, prefix_len_host, batch, block_size, bt_stride, &rows);
  if (st != CW_OK) return st;
  int64_t max_pos = -1;   // largest position of a suffix row
  for (int32_t r = 0; r < batch; ++r)
    if (cu_suffix_host[r + 1] > cu_suffix_host[r])
      max_pos = std::max<int64_t>(max_pos, int64_t(prefix_len_host[r]) + cu_suffix_host[r + 1] - cu_suffix_host[r] - 1);
  if (max_pos >= rope_len)
    return cw::fail(CW_EINVAL, std::string(what) + ": the rotary table holds " + std::to_string(rope_len) +
                                   " positions, position " + std::to_string(max_pos) + " is needed");
  if (rows == 0) return cw::ok();
  if (!x || !q_out) return cw::fail(CW_EINVAL, std::string(what) + ": x and q_out are required");
  if (rows > INT32_MAX - kTileT) return cw::fail(CW_EUNSUPPORTED, std::string(what) + ": too many suffix rows");
  const int64_t n_feat = int64_t(num_q_heads + 2 * num_kv_heads) * head_dim;
  const int64_t n_ftiles = (n_feat + kTileF - 1) / kTileF;
  const int64_t n_ttiles = (rows + kTileT - 1) / kTileT;
  const int64_t per_xcd = (n_ftiles * n_ttiles + cw::kNumXcd - 1) / cw::kNumXcd;
  if (per_xcd * cw::kNumXcd > INT32_MAX) return cw::fail(CW_EUNSUPPORTED, std::string(what) + ": too many tiles");
  auto* s = static_cast<hipStream_t>(stream);
  const dim3 grid(unsigned(per_xcd * cw::kNumXcd));
  auto* xp = static_cast<const uint8_t*>(x);
  auto* wp = static_cast<const uint8_t*>(w);
  auto* bp = static_cast<const uint16_t*>(bias);
  auto* qp = static_cast<uint16_t*>(q_out);
  auto* kp = static_cast<uint16_t*>(k_cache);
  auto* vp = static_cast<uint16_t*>(v_cache);
  if (head_dim == 128)
    hipLaunchKernelGGL(qkv_rope_append_kernel<128>, grid, dim3(kThreads), 0, s, xp, wp, bp, rope, int(rows), hidden,
                       int(n_feat), qp, kp, vp, block_table, bt_stride, cu_suffix_dev, prefix_len_dev, batch,
                       num_q_heads, num_kv_heads, num_blocks, int(n_ftiles), int(n_ttiles), int(per_xcd));
  else
    hipLaunchKernelGGL(qkv_rope_append_kernel<64>, grid, dim3(kThreads), 0, s, xp, wp, bp, rope, int(rows), hidden,
                       int(n_feat), qp, kp, vp, block_table, bt_stride, cu_suffix_dev, prefix_len_dev, batch,
                       num_q_heads, num_kv_heads, num_blocks, int(n_ftiles), int(n_ttiles), int(per_xcd));
  return check_launch("qkv_rope_append launch");
}

// Device half of libcw for gfx950 (MI355X): suffix KV append and suffix
// prefill attention over a paged, prefix-cached KV store.
//
// Paper Sec. 1 and 2.1: with a reused prefix of P cached tokens, only the S
// suffix tokens are prefilled; they attend causally over themselves and fully
// over the prefix, whose K/V the engine keeps in fixed-size blocks.
//
// Attention kernel design (one workgroup = 4 wavefronts = one tile):
//  * A tile is (request r, KV head g, a run of T suffix rows); its 128 MFMA
//    rows pack the G = Hq/Hkv query heads of g over T = 128/G positions, so
//    every K/V byte staged in LDS serves all heads of the group.
//  * Each wave owns 32 packed rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16: in the 32x32 accumulator layout a lane then
//    holds one query column and 16 keys, so row max / sum need one exchange
//    with lane ^ 32 and the softmax state (m, l, rescale) is lane-local.
//  * O^T = V^T P^T reuses the score registers directly as the B operand (the
//    key order inside an MFMA's 16-key slice only has to agree between A and
//    B); V is transposed into LDS as [d][key] when it is staged.
//  * K/V tiles of 64 keys (4 blocks) are gathered through the block table with
//    16-byte loads (each block of one KV head is one contiguous 16 x D run),
//    prefetched into registers while the previous tile is computed.
//  * Softmax in fp32 with exp2 and the scale folded into one FMA; only tiles
//    that cross the causal diagonal apply the mask; keys past the prompt end
//    are zero-filled so stale cache bytes never reach the result.

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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bfloat16 (round to nearest even) in one dword, low first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// ---------------------------------------------------------------------------
// KV append: one workgroup per suffix row. The row's request, position and
// destination block are found once per workgroup (uniform, scalar); each
// thread then moves 16-byte chunks, K first then V, so reads of k_new/v_new
// are contiguous per row and writes are contiguous per (row, head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, u32x4* __restrict__ k_cache,
    u32x4* __restrict__ v_cache, const int32_t* __restrict__ bt, int bt_stride,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ plen, int batch, int hkv,
    int chunks_per_head, int num_blocks) {
  const int row = blockIdx.x;
  // request owning this row: the largest r with cu[r] <= row
  int lo = 0, hi = batch;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= row) lo = mid; else hi = mid;
  }
  const int t = plen[lo] + (row - cu[lo]);
  const int blk = bt[int64_t(lo) * bt_stride + t / kBs];
  if (blk < 0 || blk >= num_blocks) return;
  const int per_tensor = hkv * chunks_per_head;
  const int64_t src0 = int64_t(row) * per_tensor;
  const int64_t dst0 = (int64_t(blk) * hkv * kBs + (t % kBs)) * chunks_per_head;
  for (int c = threadIdx.x; c < 2 * per_tensor; c += kThreads) {
    const int tensor = c >= per_tensor;
    const int cc = c - tensor * per_tensor;
    const int h = cc / chunks_per_head;
    const int ch = cc - h * chunks_per_head;
    const int64_t dst = dst0 + int64_t(h) * kBs * chunks_per_head + ch;
    if (tensor) v_cache[dst] = v_new[src0 + cc];
    else k_cache[dst] = k_new[src0 + cc];
  }
}

// ---------------------------------------------------------------------------
// Suffix prefill attention.
//
// LDS holds two K/V stages (double buffering, one barrier per 64-key step).
// The next step's K/V are fetched into registers while the current step is
// computed, then written into the other stage.
//  * K: row-major [key][d], rows padded by 16 bytes, so the 16-row groups of
//    the QK^T operand reads fall on distinct banks.
//  * V: row-major [key][d] with the 16-byte chunks of each row XOR-swizzled by
//    fv(row), spreading the eight rows one transposing read touches over all
//    chunk groups. V feeds the PV MFMA through ds_read_b64_tr_b16: in each
//    16-lane group, lane o receives element o % 4 of the 8-byte pieces addressed
//    by lanes o / 4 + 4 j, j = 0..3; so lane i addresses key (base + i / 4),
//    d (base + 4 (i % 4)), and lane o receives d = base + o for four keys.
// ---------------------------------------------------------------------------
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;

template <int D>
struct AttnGeom {
  static constexpr int RB = 2 * D;              // bytes per K/V row in global memory
  static constexpr int KRB = RB + 16;           // padded K row in LDS
  static constexpr int NC = D / 8;              // 16-byte chunks per row
  static constexpr int KTILE = kKv * KRB;
  static constexpr int VTILE = kKv * RB;
  static constexpr int STAGE = KTILE + VTILE;
  static constexpr int RPL = 1024 / RB;         // rows covered by one wave-wide 16-byte load
  static constexpr int LPW = kBs / RPL;         // loads per wave per tensor (one block)
  static constexpr int KS = D / 16;             // MFMA k-steps over D
  static constexpr int DT = D / 32;             // 32-row output tiles over D
  __device__ static int vswz(int row) {
    return D == 128 ? (4 * (row & 3) + ((row >> 2) & 3)) : (row & (NC - 1));
  }
};

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void suffix_prefill_attn_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
                                const uint16_t* __restrict__ vc, const int32_t* __restrict__ bt,
                                int bt_stride, const int32_t* __restrict__ cu,
                                const int32_t* __restrict__ plen, const int4* __restrict__ plan,
                                int batch, int hq, int hkv, int group, int per_tile, int num_blocks,
                                float c_log2, uint16_t* __restrict__ out) {
  using G = AttnGeom<D>;
  constexpr int KS = G::KS, DT = G::DT, RB = G::RB, KRB = G::KRB, NC = G::NC, LPW = G::LPW;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * G::STAGE];

  const int4 item = plan[blockIdx.x];
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

  bf16x8 qf[KS];
  if (row_ok) {
    const u32x4* qp = reinterpret_cast<const u32x4*>(q + (qrow * hq + head) * D);
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = __builtin_bit_cast(bf16x8, qp[2 * s + half]);
  } else {
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
  }

  // ---- K/V staging. Wave w fetches block w of each 64-key step: LPW 16-byte
  // loads per tensor per lane, lane l of load i reading row RPL i + l / NC,
  // chunk l % NC (one contiguous 1 KB run per load).
  // Physical block of logical block lb, or -1 past the prompt / outside the
  // pool; the table index is clamped into the request's row (always in bounds).
  auto block_id = [&](int lb) -> int {
    const int b = btr[min(lb, nblk - 1)];
    return (lb < nblk && b >= 0 && b < num_blocks) ? b : -1;
  };
  const int ld_row = lane / NC;
  const int ld_ch = lane % NC;
  u32x4 kreg[LPW], vreg[LPW];
  auto fetch = [&](int b) {
    const int bb = b < 0 ? 0 : b;   // block 0 stands in for a missing block; zeroed when staged
    const uint8_t* kb = reinterpret_cast<const uint8_t*>(kc) + (int64_t(bb) * hkv + g) * (kBs * RB);
    const uint8_t* vb = reinterpret_cast<const uint8_t*>(vc) + (int64_t(bb) * hkv + g) * (kBs * RB);
    const int off = ld_row * RB + ld_ch * 16;
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      kreg[i] = *reinterpret_cast<const u32x4*>(kb + off + i * 1024);
      vreg[i] = *reinterpret_cast<const u32x4*>(vb + off + i * 1024);
    }
  };
  // Rows of a missing block and rows past the prompt end are written as zeros
  // (stale cache bytes must never meet a zero probability).
  auto stage_write = [&](uint8_t* st, int k0, int b) {
    const int key0 = k0 + kBs * wave;
    if (b >= 0 && key0 + kBs <= L) {   // wave-uniform: the whole block is valid
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        const int row = kBs * wave + G::RPL * i + ld_row;
        *reinterpret_cast<u32x4*>(st + row * KRB + ld_ch * 16) = kreg[i];
        *reinterpret_cast<u32x4*>(st + G::KTILE + row * RB + ((ld_ch ^ G::vswz(row)) << 4)) = vreg[i];
      }
      return;
    }
    const u32x4 zero{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const int row = kBs * wave + G::RPL * i + ld_row;
      const bool ok = b >= 0 && key0 + G::RPL * i + ld_row < L;
      *reinterpret_cast<u32x4*>(st + row * KRB + ld_ch * 16) = ok ? kreg[i] : zero;
      *reinterpret_cast<u32x4*>(st + G::KTILE + row * RB + ((ld_ch ^ G::vswz(row)) << 4)) = ok ? vreg[i] : zero;
    }
  };

  // ---- per-lane LDS read offsets (relative to a stage)
  // K operand: row st*32 + l32, chunk 2s + half.
  const int k_off = l32 * KRB + half * 16;
  // V operand (transposing read): group gi = lane / 16, i = lane % 16:
  //   key = 16 kk + 8 sel + 4 (gi / 2) + i / 4,  d = 32 t + 16 (gi % 2) + 4 (i % 4).
  // vswz(key) depends on key mod 16 only, so kk enters as a constant offset.
  const int gi = lane >> 4, li = lane & 15;
  const int vkey_l = 4 * (gi >> 1) + (li >> 2);
  const int vd_l = 16 * (gi & 1) + 4 * (li & 3);
  int v_off[DT][2];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int sel = 0; sel < 2; ++sel) {
      const int key = 8 * sel + vkey_l;
      const int d = 32 * t + vd_l;
      v_off[t][sel] = G::KTILE + key * RB + (((d >> 3) ^ G::vswz(key)) << 4) + ((d & 4) << 1);
    }

  f32x16 oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) oacc[t] = f32x16{};
  float m_run = -INFINITY;   // running max (raw score units) used for the exponent
  float l_run = 0.f;         // this lane's partial row sum (its 32 keys per step)
  const bf16x2 ones{(__bf16)1.0f, (__bf16)1.0f};
  // Lazy rescaling: the exponent base m_run moves only when a score exceeds it
  // by more than 2^8 in probability, so O and l are rarely rescaled.
  const float lazy = 8.0f / c_log2;

  auto compute = [&](const uint8_t* st, int k0) {
    // S^T = K Q^T for keys k0 .. k0 + 63 (two 32-key halves).
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(st + k_off + h * 32 * KRB + s * 32));
        sacc[h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[h], 0, 0, 0);
      }
    // Causal mask, only where the step reaches past the first row's limit.
    if (k0 + kKv - 1 > P + row0) {
      const int lim = qpos - k0;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = h * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
          if (key > lim) sacc[h][e] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mx = fmaxf(mx, fmaxf(sacc[h][e], sacc[h][e + 1]));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // key 0 is visible to every row, so after the first step m_run is finite
    const bool grow = !(mx <= m_run + lazy);
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float m_new = grow ? fmaxf(mx, m_run) : m_run;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t) oacc[t] *= alpha;
      m_run = m_new;
    }
    const float mc = m_run * c_log2;
    bf16x8 pb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int h = kk >> 1, e0 = (kk & 1) * 8;
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[h][e0 + 2 * j], c_log2, -mc));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[h][e0 + 2 * j + 1], c_log2, -mc));
        w[j] = pack_bf16x2(p0, p1);
        l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[j]), ones, l_run, false);
      }
      pb[kk] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
    // O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const i16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4_t*)((lds_u8_t*)st + v_off[t][0] + kk * 16 * RB));
        const i16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4_t*)((lds_u8_t*)st + v_off[t][1] + kk * 16 * RB));
        const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kk], oacc[t], 0, 0, 0);
      }
  };

  // One step: fetch the next step's K/V into registers, compute this step from
  // stage SI, write the registers into the other stage, then one barrier.
  int b_next = block_id(wave);
  fetch(b_next);
  stage_write(lds, 0, b_next);
  if (ntiles > 1) b_next = block_id(kKv / kBs + wave);
  __syncthreads();
  auto step = [&](auto si, int it) {
    constexpr int SI = decltype(si)::value;
    const int k0 = it * kKv;
    const bool more = it + 1 < ntiles;
    const int b = b_next;
    if (more) {
      fetch(b);
      if (it + 2 < ntiles) b_next = block_id((k0 + 2 * kKv) / kBs + wave);
    }
    compute(lds + SI * G::STAGE, k0);
    if (more) stage_write(lds + (1 - SI) * G::STAGE, k0 + kKv, b);
    __syncthreads();
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
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
  const int cph = head_dim / 8;
  if (rows > INT32_MAX) return cw::fail(CW_EUNSUPPORTED, "kv_append: batch too large");
  hipLaunchKernelGGL(kv_append_kernel, dim3(unsigned(rows)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(k_new),
                     static_cast<const u32x4*>(v_new), static_cast<u32x4*>(k_cache),
                     static_cast<u32x4*>(v_cache), block_table, bt_stride, cu_suffix_dev,
                     prefix_len_dev, batch, num_kv_heads, cph, num_blocks);
  return check_launch("kv_append launch");
}

extern "C" cw_status cw_suffix_prefill_attn(const void* q, const void* k_cache, const void* v_cache,
                                            const int32_t* block_table, int32_t bt_stride,
                                            const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                            const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                            int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                            int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                            float softmax_scale, const int32_t* plan_dev,
                                            int32_t num_tiles, void* out, void* stream) {
  if (!q || !k_cache || !v_cache || !block_table || !cu_suffix_dev || !prefix_len_dev || !out)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn: a required pointer is NULL");
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn: num_q_heads must be a positive multiple of num_kv_heads");
  if (num_blocks < 1) return cw::fail(CW_EINVAL, "suffix_prefill_attn: num_blocks must be >= 1");
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    return cw::fail(CW_EINVAL, "suffix_prefill_attn: softmax_scale must be finite and positive");
  if (head_dim != 64 && head_dim != 128)
    return cw::fail(CW_EUNSUPPORTED, "suffix_prefill_attn: head_dim must be 64 or 128");
  if (block_size != kBs) return cw::fail(CW_EUNSUPPORTED, "suffix_prefill_attn: block_size must be 16");
  const int group = num_q_heads / num_kv_heads;
  if (group > cw::kMaxGroup)
    return cw::fail(CW_EUNSUPPORTED, "suffix_prefill_attn: more than 128 query heads per KV head");
  int64_t rows = 0;
  cw_status st = cw::check_batch(cu_suffix_host, prefix_len_host, batch, block_size, bt_stride, &rows);
  if (st != CW_OK) return st;
  const int per_tile = cw::tile_positions(group);
  const int64_t need = cw::count_tiles(cu_suffix_host, batch, num_kv_heads, per_tile);
  if (num_tiles < need || int64_t(num_tiles) > need * cw::kNumXcd)
    return cw::fail(CW_EINVAL, "suffix_prefill_attn: num_tiles " + std::to_string(num_tiles) +
                                   " does not match the batch (" + std::to_string(need) + " tiles)");
  if (num_tiles > 0 && !plan_dev) return cw::fail(CW_EINVAL, "suffix_prefill_attn: plan_dev is required");
  if (rows == 0 || num_tiles == 0) return cw::ok();
  const float c_log2 = softmax_scale * 1.4426950408889634f;
  auto* s = static_cast<hipStream_t>(stream);
  auto* qp = static_cast<const uint16_t*>(q);
  auto* kp = static_cast<const uint16_t*>(k_cache);
  auto* vp = static_cast<const uint16_t*>(v_cache);
  auto* pp = reinterpret_cast<const int4*>(plan_dev);
  auto* op = static_cast<uint16_t*>(out);
  if (head_dim == 128)
    hipLaunchKernelGGL(suffix_prefill_attn_kernel<128>, dim3(unsigned(num_tiles)), dim3(kThreads), 0, s,
                       qp, kp, vp, block_table, bt_stride, cu_suffix_dev, prefix_len_dev, pp, batch,
                       num_q_heads, num_kv_heads, group, per_tile, num_blocks, c_log2, op);
  else
    hipLaunchKernelGGL(suffix_prefill_attn_kernel<64>, dim3(unsigned(num_tiles)), dim3(kThreads), 0, s,
                       qp, kp, vp, block_table, bt_stride, cu_suffix_dev, prefix_len_dev, pp, batch,
                       num_q_heads, num_kv_heads, group, per_tile, num_blocks, c_log2, op);
  return check_launch("suffix_prefill_attn launch");
}

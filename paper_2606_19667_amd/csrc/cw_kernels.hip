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
// KV append: thread u moves 16 bytes; u enumerates (suffix row, K|V, head,
// 16-byte chunk of D), so reads of k_new/v_new are contiguous per row and
// writes are contiguous per (row, head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void kv_append_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, u32x4* __restrict__ k_cache,
    u32x4* __restrict__ v_cache, const int32_t* __restrict__ bt, int bt_stride,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ plen, int batch, int hkv,
    int chunks_per_head, int num_blocks, int64_t total_units) {
  const int64_t u = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (u >= total_units) return;
  const int per_head = chunks_per_head;
  const int per_tensor = hkv * per_head;
  const int per_row = 2 * per_tensor;
  const int row = int(u / per_row);
  int rem = int(u - int64_t(row) * per_row);
  const int tensor = rem >= per_tensor;
  rem -= tensor * per_tensor;
  const int h = rem / per_head;
  const int c = rem - h * per_head;
  // request owning this row: the largest r with cu[r] <= row
  int lo = 0, hi = batch;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= row) lo = mid; else hi = mid;
  }
  const int t = plen[lo] + (row - cu[lo]);
  const int blk = bt[int64_t(lo) * bt_stride + t / kBs];
  if (blk < 0 || blk >= num_blocks) return;
  const int64_t src = int64_t(row) * per_tensor + h * per_head + c;
  const int64_t dst = ((int64_t(blk) * hkv + h) * kBs + (t % kBs)) * per_head + c;
  if (tensor) v_cache[dst] = v_new[src];
  else k_cache[dst] = k_new[src];
}

// ---------------------------------------------------------------------------
// Suffix prefill attention.
// ---------------------------------------------------------------------------
template <int D>
struct AttnSmem {
  uint16_t k[kKv][D + 8];    // keys, row-major; 16-byte pad staggers LDS banks
  uint16_t vt[D][kKv + 4];   // values transposed to [d][key]; 8-byte pad
};

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void suffix_prefill_attn_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
                                const uint16_t* __restrict__ vc, const int32_t* __restrict__ bt,
                                int bt_stride, const int32_t* __restrict__ cu,
                                const int32_t* __restrict__ plen, const int4* __restrict__ plan,
                                int batch, int hq, int hkv, int group, int per_tile, int num_blocks,
                                float c_log2, uint16_t* __restrict__ out) {
  constexpr int CPR = D / 8;                    // 16-byte chunks per key row
  constexpr int KCH = kKv * CPR / kThreads;     // K chunks per thread per tile
  constexpr int VK = kKv * CPR / kThreads;      // consecutive V keys per thread
  constexpr int KROWS = kThreads / CPR;         // key rows covered per K chunk step
  constexpr int KS = D / 16;                    // MFMA k-steps over D
  constexpr int DT = D / 32;                    // 32-row output tiles over D
  static_assert(KCH * kThreads == kKv * CPR && VK * (kThreads / CPR) == kKv, "tile split");

  __shared__ AttnSmem<D> sm;

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
  const int32_t* btr = bt + int64_t(r) * bt_stride;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int half = lane >> 5;

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

  // Staging registers for one K/V tile.
  u32x4 ks[KCH];
  u32x4 vs[VK];
  const int dc = tid % CPR;
  const int vkey0 = (tid / CPR) * VK;

  auto block_of = [&](int key) -> int {
    if (key >= L) return -1;
    const int b = btr[key >> 4];
    return (b >= 0 && b < num_blocks) ? b : -1;
  };
  auto fetch = [&](int k0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int key = k0 + tid / CPR + KROWS * i;
      const int b = block_of(key);
      ks[i] = b < 0 ? u32x4{0, 0, 0, 0}
                    : *reinterpret_cast<const u32x4*>(
                          kc + ((int64_t(b) * hkv + g) * kBs + (key & (kBs - 1))) * D + dc * 8);
    }
#pragma unroll
    for (int j = 0; j < VK; ++j) {
      const int key = k0 + vkey0 + j;
      const int b = block_of(key);
      vs[j] = b < 0 ? u32x4{0, 0, 0, 0}
                    : *reinterpret_cast<const u32x4*>(
                          vc + ((int64_t(b) * hkv + g) * kBs + (key & (kBs - 1))) * D + dc * 8);
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i)
      *reinterpret_cast<u32x4*>(&sm.k[tid / CPR + KROWS * i][dc * 8]) = ks[i];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int d = dc * 8 + 2 * w;
      if constexpr (VK == 4) {
        const u32x2 lo{(vs[0][w] & 0xFFFFu) | (vs[1][w] << 16), (vs[2][w] & 0xFFFFu) | (vs[3][w] << 16)};
        const u32x2 hi{(vs[0][w] >> 16) | (vs[1][w] & 0xFFFF0000u), (vs[2][w] >> 16) | (vs[3][w] & 0xFFFF0000u)};
        *reinterpret_cast<u32x2*>(&sm.vt[d][vkey0]) = lo;
        *reinterpret_cast<u32x2*>(&sm.vt[d + 1][vkey0]) = hi;
      } else {
        *reinterpret_cast<uint32_t*>(&sm.vt[d][vkey0]) = (vs[0][w] & 0xFFFFu) | (vs[1][w] << 16);
        *reinterpret_cast<uint32_t*>(&sm.vt[d + 1][vkey0]) = (vs[0][w] >> 16) | (vs[1][w] & 0xFFFF0000u);
      }
    }
  };

  f32x16 oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) oacc[t] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;

  fetch(0);
  for (int it = 0; it < ntiles; ++it) {
    const int k0 = it * kKv;
    __syncthreads();
    stage();
    __syncthreads();
    if (it + 1 < ntiles) fetch(k0 + kKv);

    // S^T = K Q^T for keys k0 .. k0+63 (two 32-key halves).
    f32x16 sacc[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      sacc[st] = f32x16{};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sm.k[st * 32 + l32][s * 16 + half * 8]));
        sacc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[st], 0, 0, 0);
      }
    }

    // Causal mask, only where the tile reaches past the first row's limit.
    if (k0 + kKv - 1 > P + row0) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = k0 + st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
          if (key > qpos) sacc[st][e] = -INFINITY;
        }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[st][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);          // finite: key 0 is visible to every row
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
    const float mc = m_new * c_log2;
    float lsum = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[st][e], c_log2, -mc));
        sacc[st][e] = p;
        lsum += p;
      }
    l_run = l_run * alpha + lsum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < DT; ++t) oacc[t] *= alpha;

    // P^T as the B operand: slice kk holds keys 16kk .. 16kk+15.
    bf16x8 pb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int st = kk >> 1, e0 = (kk & 1) * 8;
      const u32x4 w{pack_bf16x2(sacc[st][e0 + 0], sacc[st][e0 + 1]),
                    pack_bf16x2(sacc[st][e0 + 2], sacc[st][e0 + 3]),
                    pack_bf16x2(sacc[st][e0 + 4], sacc[st][e0 + 5]),
                    pack_bf16x2(sacc[st][e0 + 6], sacc[st][e0 + 7])};
      pb[kk] = __builtin_bit_cast(bf16x8, w);
    }

    // O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const uint16_t* vrow = &sm.vt[t * 32 + l32][16 * kk + 4 * half];
        const u32x2 a0 = *reinterpret_cast<const u32x2*>(vrow);
        const u32x2 a1 = *reinterpret_cast<const u32x2*>(vrow + 8);
        const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{a0[0], a0[1], a1[0], a1[1]});
        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kk], oacc[t], 0, 0, 0);
      }
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
  const int64_t units = rows * 2 * num_kv_heads * cph;
  const int64_t grid = (units + kThreads - 1) / kThreads;
  if (grid > INT32_MAX) return cw::fail(CW_EUNSUPPORTED, "kv_append: batch too large");
  hipLaunchKernelGGL(kv_append_kernel, dim3(unsigned(grid)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(k_new),
                     static_cast<const u32x4*>(v_new), static_cast<u32x4*>(k_cache),
                     static_cast<u32x4*>(v_cache), block_table, bt_stride, cu_suffix_dev,
                     prefix_len_dev, batch, num_kv_heads, cph, num_blocks, units);
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
  if (group > cw::kTileRows)
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

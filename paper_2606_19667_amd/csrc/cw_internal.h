// Internal declarations shared by the host and device translation units of libcw.
#pragma once

#include <cstdint>
#include <string>

#ifndef __HIPCC__
#define __host__
#define __device__
#endif

#include "cw.h"

namespace cw {

// Records `msg` as the calling thread's last error and returns `status`.
cw_status fail(cw_status status, const std::string& msg);
// Clears the calling thread's last error and returns CW_OK.
cw_status ok();

// Tile geometry of the attention kernel, shared with the planner.
constexpr int kBlockSize = 16;   // tokens per KV block
constexpr int kTileRows = 256;   // packed query rows (heads x positions) per workgroup
constexpr int kKvTile = 64;      // keys staged in LDS per step
constexpr int kNumXcd = 8;       // L2 partitions; workgroup i runs on partition i % 8
constexpr int kMaxGroup = 128;   // query heads per KV head supported
constexpr int kMaxKvHeads = 65536;   // KV heads supported by the attention calls

constexpr int kNumCu = 256;      // compute units: the attention grid's persistent workgroups
constexpr int kMaxSplits = 64;   // key runs per tile on the split path
constexpr int64_t kNoAllocScratchBytes = int64_t(64) << 20;   // scratch of the allocation-free split call

// Suffix positions covered by one tile for a GQA group of `group` query heads.
inline int tile_positions(int group) { return kTileRows / group; }

// Attention plan layout (int32 words), written by cw_suffix_prefill_plan and
// read by the attention kernels: a header, then entries of kPlanEntryWords.
constexpr int kPlanHeaderWords = 16;
constexpr int kPlanEntryWords = 16;
constexpr int32_t kPlanMagic = 0x33505743;   // "CWP3"
// header words
constexpr int kHdrMagic = 0, kHdrEntries = 1, kHdrFpLo = 2, kHdrFpHi = 3, kHdrGrid = 4, kHdrSplits = 5,
              kHdrBatch = 6, kHdrHq = 7, kHdrHkv = 8, kHdrD = 9, kHdrRows = 10, kHdrQueueLen = 11,
              kHdrWork = 12, kHdrTable = 13, kHdrTableStride = 14, kHdrNumBlocks = 15;
// A plan for the fused append + attention call (cw_suffix_prefill_append_plan)
// also holds, at word kHdrTable (0 in other plans), a block table of pairs:
// for request r and logical block j, words [r][j][0..1] at stride
// kHdrTableStride pairs per request are
//   source:      16 b for cache block b; 0x80000000 | R for rows R .. R + 15
//                of k_new / v_new; -1 no block (zeros). The kernel scales the
//                low 31 bits by the bytes of one k_new row (Hkv rows of D):
//                a cache block is 16 such rows.
//   destination: the cache block the entry owning the block's rows writes
//                them to (a suffix block of this call), else -1
// entry words: request (-1 ends a queue), KV head, first suffix row, rows,
// the request's first row in q/out, its prefix and prompt lengths, the run of
// 64-key steps [kbeg, kend), the run's index, the number of the run's steps
// (from kbeg) that every row sees whole (no causal mask), the entry's first
// row in q/out, and a check word
constexpr int kEntR = 0, kEntG = 1, kEntRow0 = 2, kEntNvalid = 3, kEntCu0 = 4, kEntP = 5, kEntL = 6,
              kEntKbeg = 7, kEntKend = 8, kEntSplit = 9, kEntNfull = 10, kEntQrow = 11, kEntCheck = 15;
constexpr int kEntFields = 12;   // words the planner fills besides the check word
// source words of the fused plan's table
constexpr int32_t kMaxAppendBlocks = (1 << 27) - 1;   // pool blocks a fused plan supports (16 b < 2^31)
inline int32_t append_src_block(int32_t b) { return 16 * b; }
inline int32_t append_src_rows(int32_t row) { return int32_t(0x80000000u | uint32_t(row)); }

// Check word of the plan entry at position `index` of a plan body: derived
// from the batch fingerprint and the position. The planner is deterministic,
// so an entry whose word matches was written, at that position, by a plan for
// this batch; the kernels end a queue at an entry that does not match (e.g.
// entries of an earlier plan left behind a newer header in device memory).
__host__ __device__ inline uint32_t entry_tag(uint32_t fp_lo, uint32_t fp_hi, uint32_t index) {
  return (fp_lo ^ (index * 0x9E3779B1u)) + fp_hi;
}

// 64-bit fingerprint of a batch description as a plan is built for it.
uint64_t batch_fingerprint(const int32_t* cu_suffix_host, const int32_t* prefix_len_host, int32_t batch,
                           int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t num_splits);
// Fingerprint of a fused plan: the batch fingerprint (one split) mixed with the
// block table words of every request's prompt blocks and the pool size.
uint64_t append_fingerprint(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                            const int32_t* block_table_host, int32_t bt_stride, int32_t batch, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, int32_t num_blocks);

// Validates the ragged batch description shared by the device entry points.
// Checks cu[0] == 0, cu non-decreasing, P_r >= 0 and a multiple of
// block_size, ceil(L_r / block_size) <= bt_stride; sets *total_rows.
cw_status check_batch(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                      int32_t batch, int32_t block_size, int32_t bt_stride,
                      int64_t* total_rows);

// Number of (request, kv head, row run) tiles of a batch, before padding.
int64_t count_tiles(const int32_t* cu_suffix_host, int32_t batch, int32_t num_kv_heads,
                    int32_t positions_per_tile);

// Checks a plan's header (plan_host, as cw_suffix_prefill_plan wrote it)
// against the batch description of a device call: magic, fingerprint of
// cu / prefix_len / heads / head_dim / split count, queue geometry. Sets the
// launch grid, the split count, the fingerprint words and the entry count.
// For the fused call (append_bt set: the host block table, its stride and
// the pool size) the plan must carry an append table built for that table;
// for the other calls it must not carry one.
cw_status check_plan_header(const char* what, const int32_t* plan_host, const int32_t* cu, const int32_t* plen,
                            int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t* grid, int32_t* splits,
                            uint32_t* fp_lo, uint32_t* fp_hi, int32_t* num_entries,
                            const int32_t* append_bt = nullptr, int32_t bt_stride = 0, int32_t num_blocks = 0);

}  // namespace cw

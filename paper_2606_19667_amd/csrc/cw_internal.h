// Internal declarations shared by the host and device translation units of libcw.
#pragma once

#include <cstdint>
#include <string>

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

// Suffix positions covered by one tile for a GQA group of `group` query heads.
inline int tile_positions(int group) { return kTileRows / group; }

// Validates the ragged batch description shared by the device entry points.
// Checks cu[0] == 0, cu non-decreasing, P_r >= 0 and a multiple of
// block_size, ceil(L_r / block_size) <= bt_stride; sets *total_rows.
cw_status check_batch(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                      int32_t batch, int32_t block_size, int32_t bt_stride,
                      int64_t* total_rows);

// Number of (request, kv head, row run) tiles of a batch, before padding.
int64_t count_tiles(const int32_t* cu_suffix_host, int32_t batch, int32_t num_kv_heads,
                    int32_t positions_per_tile);

}  // namespace cw

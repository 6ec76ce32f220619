// Constants and table formats shared by the host code and the HIP kernels of libra:
// everything the device code reads from the plan workspace is laid out here.
#pragma once

#include <cstdint>

#include "libra.h"

namespace libra {

constexpr int kPage = LIBRA_PAGE_SIZE;     // tokens per page
constexpr int kDim = LIBRA_HEAD_DIM;       // channels per head
constexpr int kTileElems = kPage * kDim;   // bf16 elements per (page, head) tile
constexpr int kTileBytes = kTileElems * 2; // 4 KiB
constexpr int kUnitInts = LIBRA_UNIT_INTS;

// Unit record fields (int32), in table order.
enum UnitField : int {
  U_B = 0, U_G, U_KV0, U_KV1, U_Q0, U_Q1, U_SPLIT, U_NSPLIT, U_PART, U_ROW0, U_KIND, U_PRIOR
};
constexpr int kKindSingle = 0;
constexpr int kKindChunk = 1;
constexpr int kNumXcds = 8;  // MI355X: workgroup w is dispatched to XCD w % 8
constexpr int kChunkStepKeys = 64;  // keys per step of the chunk kernel's key loop
constexpr int kChunkRows = 256;  // (token, head) rows of one chunk-kernel tile

// Append cache-write table: one record per (sequence, page) the new tokens touch.
enum WriteField : int { W_B = 0, W_PAGE, W_SLOT0, W_SLOT1, W_ROW, W_PAD0, W_PAD1, W_PAD2 };
constexpr int kWriteInts = 8;

// Split-merge table: one record per (sequence, KV head) whose KV range was split.
enum MergeField : int { M_B = 0, M_G, M_N, M_PART, M_ROW, M_PAD0, M_PAD1, M_PAD2 };
constexpr int kMergeInts = 8;

}  // namespace libra

// Internal layout shared by the host plan builder (pfx_plan.cpp) and the
// device code (pfx_kernels.hip).  Not part of the public interface.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/pfx_attn.h"

namespace pfx {

// Columns of one MFMA tile: the query side of a 16x16x32 bf16 product.
constexpr int kTileCols = 16;
// Waves per phase-A workgroup; each owns 16 (decode) or 32 (extend) columns.
constexpr int kTileWaves = 4;
// Query columns of a phase-A item: decode prefix pieces and early suffix
// chunks, and extend blocks.
constexpr int kDecodeTileCols = kTileWaves * 16;
constexpr int kExtendTileCols = kTileWaves * 32;
// Page ids one phase-A item may reference (its LDS page table).
constexpr int kMaxTilePages = 1024;
// Keys processed per inner step (two 16-token pages).
constexpr int kStepKeys = 32;

enum ItemKind : int32_t { kPrefixItem = 0, kSuffixItem = 1, kExtendItem = 2 };

// One unit of device work, run by one workgroup.  Its query columns are
// row_count tokens (row_tok[row_begin ...]) times the G query heads of KV
// head kv_head.  Keys come from up to two segments of the plan's page list:
//   segment 0 (no mask):  keys [s0_kbeg, s0_kend) of the list at s0_page_off;
//   segment 1 (causal):   keys [s1_kbeg, s1_kend) of the list at s1_page_off,
//                         key k visible to token t iff k <= t + causal_base.
// out_slot >= 0: partial slot out_slot of every request the item covers;
// out_slot < 0: final rows (extend items, and decode rows whose keys one
// item covers entirely).
// tok0 >= 0: the item's tokens are tok0, tok0 + 1, ... (one request), so
// row_tok need not be read.  first_pages: the first kItemPages page ids of
// the item's keys in order (segment 0's pages, then segment 1's), so the
// first steps can be requested before the rest of the page list arrives.
constexpr int kItemPages = 16;
struct alignas(16) Item {
  int32_t kv_head;
  int32_t row_begin;
  int32_t row_count;
  int32_t nblk;
  int32_t s0_page_off, s0_kbeg, s0_kend;
  int32_t s1_page_off, s1_kbeg, s1_kend;
  int32_t causal_base;
  int32_t out_slot;
  int32_t kind;
  int32_t req;  // request of a suffix/extend item, -1 for prefix items
  int32_t tok0;
  int32_t pad0;
  int32_t first_pages[kItemPages];
};
static_assert(sizeof(Item) == 128, "Item is 32 int32");

// Per-request bookkeeping on the device.
struct ReqInfo {
  int32_t q_start;    // first query row
  int32_t n;          // query rows
  int32_t nparts;     // partial results of each row, merged last (0: rows written directly)
  int32_t part_base;  // partial row of (slot, row i): part_base + slot * n + i
};

// Device pointers into an uploaded workspace.
struct DevPlan {
  const Item* items;
  const int32_t* row_tok;
  const int32_t* page_list;
  const int32_t* tok_req;
  const ReqInfo* req;
  const int32_t* tok_slot;  // page * 16 + slot of every new token (append)
  const int32_t* merge_tok; // tokens whose rows merge several partial results
  float* o_part;            // [num_part_rows][hq][d]
  float* l_part;            // [num_part_rows][hq]
};

}  // namespace pfx

struct pfx_plan {
  int32_t num_pages = 0, hkv = 0, d = 0, hq = 0, group = 0, mode = 0;
  int32_t num_reqs = 0, num_tokens = 0;
  // items[0, n_decode): decode pieces (prefix chunks and suffix chunks,
  // writing partials or single-piece rows); then n_extend extend blocks.
  int32_t n_decode = 0, n_extend = 0;
  std::vector<int32_t> merge_tok;  // tokens whose rows merge several pieces
  std::vector<pfx::Item> items;
  std::vector<int32_t> row_tok, page_list, tok_req, tok_slot;
  std::vector<pfx::ReqInfo> req;
  int64_t num_part_rows = 0;
  int32_t n_prefix_items = 0, n_suffix_items = 0, n_extend_items = 0;
  int32_t pages_needed = 0;
  // byte offsets inside the workspace
  size_t off_items = 0, off_row_tok = 0, off_page_list = 0, off_tok_req = 0, off_req = 0,
         off_tok_slot = 0, off_merge_tok = 0, off_opart = 0, off_lpart = 0, total_bytes = 0, blob_bytes = 0;
  std::vector<unsigned char> blob;  // host image of [0, blob_bytes)
  void* dev_ws = nullptr;
  size_t dev_ws_bytes = 0;
};

namespace pfx {
// Thread-local error text, set by every failing entry point.
int fail(int code, const char* fmt, ...);
void clear_error();
pfx::DevPlan dev_plan(const pfx_plan* p);
}  // namespace pfx

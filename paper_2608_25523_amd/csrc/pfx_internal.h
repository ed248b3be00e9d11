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
// Waves per workgroup of the attention kernels.
constexpr int kTileWaves = 4;
// Query columns of a decode prefix item (16 per wave) and of an extend
// block (32 per wave).
constexpr int kDecodeTileCols = kTileWaves * 16;
constexpr int kExtendTileCols = kTileWaves * 32;
// Keys processed per inner step (two 16-token pages).
constexpr int kStepKeys = 32;

enum ItemKind : int32_t { kPrefixItem = 0, kSuffixItem = 1, kExtendItem = 2 };

// One block of query columns run by one workgroup with 32 columns per wave.
// Its columns are row_count tokens (row_tok[row_begin ...]) times the G
// query heads of KV head kv_head.  Keys come from two segments of the
// plan's page list:
//   segment 0 (no mask):  keys [s0_kbeg, s0_kend) of the list at s0_page_off;
//   segment 1 (causal):   keys [s1_kbeg, s1_kend) of the list at s1_page_off,
//                         key k visible to token t iff k <= t + causal_base.
// kind kExtendItem: an extend block; its rows are written final
// (out_slot = -1) and its tokens are tok0, tok0 + 1, ... (one request).
// kind kPrefixItem: a wide prefix block, one piece of an agent's prefix
// (segment 0 only) against up to 128 of the agent's decode columns; its
// tokens are row_tok[row_begin + j] (tok0 = -1) and it leaves partial states
// (out_slot = its slot) at partial rows row_out[row_begin + j] + g.
// first_pages: the first kItemPages page ids of the keys in order (segment
// 0's pages, then segment 1's), so the first steps can be requested before
// the rest of the page list arrives.
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
  int32_t req;
  int32_t tok0;
  int32_t pad0;
  int32_t first_pages[kItemPages];
};
static_assert(sizeof(Item) == 128, "Item is 32 int32");

// Decode work.  A decode item is one KV head's whole key range for a set of
// query rows: an agent's prefix against a block of its decode rows (<= 64
// columns), or one request's suffix against its own rows.  Items are cut
// into 32-key steps and then into pieces of at most kPieceSteps steps; each
// piece leaves its unnormalised state for the merge.  Pieces are stored
// longest first and dealt to the persistent workgroups in rounds (forward,
// then backward), so the longest run first and the shortest fill the tail.
constexpr int kSegRows = kDecodeTileCols;  // rows of a piece (columns / G)
constexpr int kPieceSteps = 64;            // steps of a piece, at most
constexpr int kPieceSlots = 4;             // pieces a workgroup holds in LDS

struct alignas(16) SegHead {
  int32_t kind;         // kPrefixItem or kSuffixItem
  int32_t kv_head;
  int32_t ncols;        // query columns: rows * G (<= 64)
  int32_t nsteps;       // 32-key steps of the piece (<= kPieceSteps)
  int32_t k0;           // key of the first step, within the item
  int32_t kend;         // keys of the item (the last step is masked past it)
  int32_t causal_base;  // suffix items: key k visible to token t iff k <= t + causal_base
  int32_t slot;         // partial slot of the piece in each of its rows; -1: final rows
  int32_t item;         // decode item
  int32_t piece;        // index of the piece within its item
  int32_t causal;       // 1: some row sees only part of the keys (multi-row suffix)
  int32_t pad[5];
};
// One piece as stored in the workspace and, unchanged, in a workgroup's LDS
// slot.
struct alignas(16) Seg {
  SegHead h;
  int32_t tok[kSegRows];          // query token of row j
  int32_t out[kSegRows];          // row j, query head g -> output row out[j] + g:
                                  // o/lse row (final) or o_part/l_part row (partial)
  int32_t steps[2 * kPieceSteps]; // per step: (page * Hkv + head) of its two 16-key pages
};
static_assert(sizeof(Seg) == 1088, "Seg is 272 int32");

// Partial results of one (decode token, KV head): nparts slots of G rows at
// o_part/l_part rows (base + slot) * G + g.  A partial row holds a piece's
// state: in l_part the pair (m, l) of its running maximum (log2 units,
// scaled) and its sum of 2^(s - m), in o_part its D accumulators
// sum_k 2^(s_k - m) v_k divided by l, as bf16.  The D * G elements of a
// slot's rows hold 16-byte units in unit-major order: unit u = 4 p + grp of
// row g (dims 32 p + 4 grp .. + 3, then 32 p + 16 + 4 grp .. + 3) at
// element (u G + g) 8, so that a wave stores each token's G rows as one
// contiguous run.
struct MergeHead {
  int32_t base;
  int32_t nparts;
};

// Device pointers into an uploaded workspace.
struct DevPlan {
  const Item* items;            // extend blocks, then wide prefix blocks
  const int32_t* row_tok;
  const int32_t* row_out;       // partial row base of each row of a wide prefix block
  const int32_t* page_list;
  const int32_t* tok_slot;      // page * 16 + slot of every new token (append)
  const Seg* segs;              // decode pieces, longest first
  const int32_t* merge_tok;     // decode tokens (their rows are merged from pieces)
  const MergeHead* merge_head;  // [merge token][KV head]
  uint16_t* o_part;             // [partial row][d] bf16, in the partial layout
  float* l_part;                // [partial row][2]
};

// Per-request bookkeeping (host).
struct ReqInfo {
  int32_t q_start;  // first query row
  int32_t n;        // query rows
};

}  // namespace pfx

struct pfx_plan {
  int32_t num_pages = 0, hkv = 0, d = 0, hq = 0, group = 0, mode = 0;
  int32_t decode_workers = 0;  // decode workgroups requested (0: one per piece)
  int32_t decode_engine = 0;   // PFX_DECODE_MFMA or PFX_DECODE_VALU
  int32_t num_reqs = 0, num_tokens = 0;
  int32_t num_items = 0;       // extend blocks (their records live in the blob at off_items)
  int32_t num_wide = 0;        // wide prefix blocks, after the extend blocks in the same array
  std::vector<int32_t> row_tok, row_out, page_list, tok_req, tok_slot;
  std::vector<pfx::ReqInfo> req;
  int32_t num_segs = 0;        // decode pieces (their records live in the blob at off_segs)
  int32_t merge_parts = 0;     // P when every merged (row, KV head) has P parts at slots (row * Hkv + h) * P, else 0
  int32_t merge_tok_is_row = 0;  // 1 when merge row m is decode token m for every m
  int64_t num_decode_steps = 0;
  std::vector<int32_t> merge_tok;
  std::vector<pfx::MergeHead> merge_head;
  int64_t num_part_rows = 0;
  int32_t n_prefix_items = 0, n_suffix_items = 0, n_extend_items = 0;
  int32_t pages_needed = 0;
  // byte offsets inside the workspace
  size_t off_items = 0, off_row_tok = 0, off_row_out = 0, off_page_list = 0, off_tok_slot = 0, off_segs = 0,
         off_merge_tok = 0, off_merge_head = 0, off_opart = 0, off_lpart = 0, total_bytes = 0, blob_bytes = 0;
  std::vector<unsigned char> blob;  // host image of [0, blob_bytes)
  const pfx::Item* host_items() const { return reinterpret_cast<const pfx::Item*>(blob.data() + off_items); }
  const pfx::Seg* host_segs() const { return reinterpret_cast<const pfx::Seg*>(blob.data() + off_segs); }
  void* dev_ws = nullptr;
  size_t dev_ws_bytes = 0;
};

namespace pfx {
// Thread-local error text, set by every failing entry point.
int fail(int code, const char* fmt, ...);
void clear_error();
// Device pointers of the plan's tables and partial states in a copy of its
// workspace image at `base` (the uploaded workspace by default).
pfx::DevPlan dev_plan(const pfx_plan* p, void* base);
inline pfx::DevPlan dev_plan(const pfx_plan* p) { return dev_plan(p, p->dev_ws); }
}  // namespace pfx

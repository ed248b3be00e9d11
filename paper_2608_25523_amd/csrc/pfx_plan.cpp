// Host side of the library: errors, the page allocator, validation and the
// plan builder.  No HIP calls live here, so this file also builds with g++
// for host-only sanitizer runs.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <unordered_map>
#include <vector>

#include "pfx_internal.h"

namespace pfx {

static thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

void clear_error() { g_err.clear(); }

// One host image kept per thread for the next plan (see pfx_plan_destroy).
static std::vector<unsigned char>& spare_blob() {
  thread_local std::vector<unsigned char> spare;
  return spare;
}

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

static int64_t pages_for(int64_t tokens) { return (tokens + PFX_PAGE_SIZE - 1) / PFX_PAGE_SIZE; }

// Longest decode piece by default, in steps: 16, or 64 once the decode
// items hold at least kLongPiecesFrom steps.  Every piece costs a Q stage,
// a partial state and its share of the merge; shorter pieces balance a
// small launch better.
constexpr int32_t kDefaultPieceSteps = 16;
constexpr int32_t kLongPieceSteps = 64;
constexpr int64_t kLongPiecesFrom = 32768;

DevPlan dev_plan(const pfx_plan* p, void* ws) {
  unsigned char* base = static_cast<unsigned char*>(ws);
  DevPlan d;
  d.items = reinterpret_cast<const Item*>(base + p->off_items);
  d.row_tok = reinterpret_cast<const int32_t*>(base + p->off_row_tok);
  d.row_out = reinterpret_cast<const int32_t*>(base + p->off_row_out);
  d.page_list = reinterpret_cast<const int32_t*>(base + p->off_page_list);
  d.tok_slot = reinterpret_cast<const int32_t*>(base + p->off_tok_slot);
  d.segs = reinterpret_cast<const Seg*>(base + p->off_segs);
  d.merge_tok = reinterpret_cast<const int32_t*>(base + p->off_merge_tok);
  d.merge_head = reinterpret_cast<const MergeHead*>(base + p->off_merge_head);
  d.o_part = reinterpret_cast<uint16_t*>(base + p->off_opart);
  d.l_part = reinterpret_cast<float*>(base + p->off_lpart);
  return d;
}

}  // namespace pfx

using pfx::fail;

extern "C" int pfx_version(void) { return PFX_VERSION; }

extern "C" const char* pfx_last_error(void) { return pfx::g_err.c_str(); }

// ---------------------------------------------------------------------------
// Page allocator
// ---------------------------------------------------------------------------

struct pfx_alloc {
  int32_t num_pages = 0;
  std::vector<int32_t> free_list;  // back() is handed out next
  std::vector<uint8_t> used;
};

extern "C" int pfx_alloc_create(int32_t num_pages, pfx_alloc** out) {
  if (!out) return fail(PFX_EINVAL, "pfx_alloc_create: out is NULL");
  *out = nullptr;
  if (num_pages < 0) return fail(PFX_ERANGE, "pfx_alloc_create: num_pages %d < 0", num_pages);
  pfx_alloc* a = new (std::nothrow) pfx_alloc;
  if (!a) return fail(PFX_ENOMEM, "pfx_alloc_create: host allocation failed");
  a->num_pages = num_pages;
  a->free_list.resize(num_pages);
  for (int32_t i = 0; i < num_pages; ++i) a->free_list[i] = num_pages - 1 - i;
  a->used.assign(num_pages, 0);
  *out = a;
  return PFX_OK;
}

extern "C" int pfx_alloc_pages(pfx_alloc* a, int32_t n, int32_t* out_ids) {
  if (!a) return fail(PFX_EINVAL, "pfx_alloc_pages: allocator is NULL");
  if (n < 0) return fail(PFX_ERANGE, "pfx_alloc_pages: n %d < 0", n);
  if (n > 0 && !out_ids) return fail(PFX_EINVAL, "pfx_alloc_pages: out_ids is NULL");
  if (static_cast<size_t>(n) > a->free_list.size())
    return fail(PFX_ENOMEM, "pfx_alloc_pages: %d pages requested, %zu free", n, a->free_list.size());
  for (int32_t i = 0; i < n; ++i) {
    int32_t id = a->free_list.back();
    a->free_list.pop_back();
    a->used[id] = 1;
    out_ids[i] = id;
  }
  return PFX_OK;
}

extern "C" int pfx_free_pages(pfx_alloc* a, const int32_t* ids, int32_t n) {
  if (!a) return fail(PFX_EINVAL, "pfx_free_pages: allocator is NULL");
  if (n < 0) return fail(PFX_ERANGE, "pfx_free_pages: n %d < 0", n);
  if (n > 0 && !ids) return fail(PFX_EINVAL, "pfx_free_pages: ids is NULL");
  std::vector<uint8_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    int32_t id = ids[i];
    if (id < 0 || id >= a->num_pages) return fail(PFX_EINVAL, "pfx_free_pages: id %d out of range", id);
    if (!a->used[id]) return fail(PFX_EINVAL, "pfx_free_pages: page %d is not allocated", id);
    if (seen.empty()) seen.assign(a->num_pages, 0);
    if (seen[id]) return fail(PFX_EINVAL, "pfx_free_pages: page %d freed twice", id);
    seen[id] = 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    a->used[ids[i]] = 0;
    a->free_list.push_back(ids[i]);
  }
  return PFX_OK;
}

extern "C" int pfx_alloc_num_free(const pfx_alloc* a, int32_t* out) {
  if (!a || !out) return fail(PFX_EINVAL, "pfx_alloc_num_free: NULL argument");
  *out = static_cast<int32_t>(a->free_list.size());
  return PFX_OK;
}

extern "C" void pfx_alloc_destroy(pfx_alloc* a) { delete a; }

// ---------------------------------------------------------------------------
// Plan
// ---------------------------------------------------------------------------

namespace {


int check_pool_shape(const pfx_pool* pool, const char* who) {
  if (!pool) return fail(PFX_EINVAL, "%s: pool is NULL", who);
  if (pool->page_size != PFX_PAGE_SIZE)
    return fail(PFX_EUNSUPPORTED, "%s: page_size %d (only %d is supported)", who, pool->page_size,
                PFX_PAGE_SIZE);
  if (pool->head_dim != 64 && pool->head_dim != 128)
    return fail(PFX_EUNSUPPORTED, "%s: head_dim %d (64 or 128 supported)", who, pool->head_dim);
  if (pool->num_kv_heads < 1) return fail(PFX_EINVAL, "%s: num_kv_heads %d < 1", who, pool->num_kv_heads);
  if (pool->num_pages < 0) return fail(PFX_ERANGE, "%s: num_pages %d < 0", who, pool->num_pages);
  return PFX_OK;
}

bool is_group_supported(int32_t g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

}  // namespace

extern "C" int pfx_plan_create(const pfx_pool* pool, const pfx_prefix_table* pt, const pfx_batch* b,
                               int32_t hq, int32_t mode, const pfx_plan_opts* opts, pfx_plan** out) {
  using namespace pfx;
  if (!out) return fail(PFX_EINVAL, "pfx_plan_create: out is NULL");
  *out = nullptr;
  int rc = check_pool_shape(pool, "pfx_plan_create");
  if (rc) return rc;
  if (!pt || !b) return fail(PFX_EINVAL, "pfx_plan_create: prefix table or batch is NULL");
  const int32_t hkv = pool->num_kv_heads;
  if (hq < 1 || hq % hkv != 0)
    return fail(PFX_EINVAL, "pfx_plan_create: num_q_heads %d is not a multiple of num_kv_heads %d", hq, hkv);
  const int32_t G = hq / hkv;
  if (!is_group_supported(G))
    return fail(PFX_EUNSUPPORTED, "pfx_plan_create: query group %d (1, 2, 4, 8 or 16 supported)", G);
  if (mode != PFX_MODE_EXTEND && mode != PFX_MODE_DECODE && mode != PFX_MODE_MIXED)
    return fail(PFX_EINVAL, "pfx_plan_create: mode %d", mode);
  int32_t p_workers = 0, piece_steps = 0, engine = PFX_DECODE_MFMA;
  if (opts) {
    for (int i = 0; i < 5; ++i)
      if (opts->reserved[i]) return fail(PFX_EINVAL, "pfx_plan_create: opts.reserved[%d] != 0", i);
    if (opts->decode_workers < 0 || opts->decode_workers > (1 << 20))
      return fail(PFX_EINVAL, "pfx_plan_create: decode_workers %d outside [0, %d]", opts->decode_workers, 1 << 20);
    if (opts->piece_steps < 0 || opts->piece_steps > kPieceSteps)
      return fail(PFX_EINVAL, "pfx_plan_create: piece_steps %d outside [0, %d]", opts->piece_steps, kPieceSteps);
    if (opts->decode_engine != PFX_DECODE_MFMA && opts->decode_engine != PFX_DECODE_VALU)
      return fail(PFX_EINVAL, "pfx_plan_create: decode_engine %d is neither PFX_DECODE_MFMA nor PFX_DECODE_VALU",
                  opts->decode_engine);
    p_workers = opts->decode_workers;
    engine = opts->decode_engine;
    if (opts->piece_steps) piece_steps = opts->piece_steps;
  }
  if (int64_t(pool->num_pages) * hkv > INT32_MAX)
    return fail(PFX_EUNSUPPORTED, "pfx_plan_create: num_pages * num_kv_heads must stay below 2^31");

  // ---- prefix table ----
  const int32_t A = pt->num_agents;
  if (A < 0) return fail(PFX_ERANGE, "pfx_plan_create: num_agents %d < 0", A);
  if (A > 0 && (!pt->page_indptr || !pt->prefix_len))
    return fail(PFX_EINVAL, "pfx_plan_create: prefix table arrays are NULL");
  if (A > 0 && pt->page_indptr[0] != 0) return fail(PFX_EINVAL, "pfx_plan_create: page_indptr[0] != 0");
  for (int32_t a = 0; a < A; ++a) {
    if (pt->prefix_len[a] < 0) return fail(PFX_ERANGE, "pfx_plan_create: prefix_len[%d] = %d", a, pt->prefix_len[a]);
    int64_t cnt = int64_t(pt->page_indptr[a + 1]) - pt->page_indptr[a];
    if (cnt != pages_for(pt->prefix_len[a]))
      return fail(PFX_EINVAL, "pfx_plan_create: agent %d has %lld pages for %d tokens (need %lld)", a,
                  (long long)cnt, pt->prefix_len[a], (long long)pages_for(pt->prefix_len[a]));
  }
  if (A > 0 && pt->page_indptr[A] > 0 && !pt->page_ids)
    return fail(PFX_EINVAL, "pfx_plan_create: page_ids is NULL");

  // ---- batch ----
  const int32_t R = b->num_reqs;
  if (R < 0) return fail(PFX_ERANGE, "pfx_plan_create: num_reqs %d < 0", R);
  if (R > 0 && (!b->agent || !b->suffix_indptr || !b->suffix_len || !b->q_indptr))
    return fail(PFX_EINVAL, "pfx_plan_create: batch arrays are NULL");
  if (R > 0 && (b->suffix_indptr[0] != 0 || b->q_indptr[0] != 0))
    return fail(PFX_EINVAL, "pfx_plan_create: suffix_indptr[0] and q_indptr[0] must be 0");
  int64_t total_tokens = 0;
  for (int32_t r = 0; r < R; ++r) {
    int32_t L = b->suffix_len[r];
    if (L < 0) return fail(PFX_ERANGE, "pfx_plan_create: suffix_len[%d] = %d", r, L);
    int64_t cnt = int64_t(b->suffix_indptr[r + 1]) - b->suffix_indptr[r];
    if (cnt != pages_for(L))
      return fail(PFX_EINVAL, "pfx_plan_create: request %d has %lld suffix pages for %d tokens", r, (long long)cnt, L);
    int64_t n = int64_t(b->q_indptr[r + 1]) - b->q_indptr[r];
    if (n < 0) return fail(PFX_EINVAL, "pfx_plan_create: q_indptr decreases at request %d", r);
    if (n > L) return fail(PFX_ERANGE, "pfx_plan_create: request %d has %lld query rows but suffix_len %d", r, (long long)n, L);
    if (mode == PFX_MODE_DECODE && n > 1)
      return fail(PFX_EINVAL, "pfx_plan_create: decode mode but request %d has %lld query rows", r, (long long)n);
    int32_t a = b->agent[r];
    if (a < -1 || a >= A) return fail(PFX_ERANGE, "pfx_plan_create: agent[%d] = %d (num_agents %d)", r, a, A);
    total_tokens += n;
  }
  if (total_tokens > (int64_t(1) << 30)) return fail(PFX_ERANGE, "pfx_plan_create: too many query rows");
  if (R > 0 && b->suffix_indptr[R] > 0 && !b->suffix_page_ids)
    return fail(PFX_EINVAL, "pfx_plan_create: suffix_page_ids is NULL");

  // ---- Sec. 3, Eq. (2): prefixes counted once, plus every request's own KV ----
  std::vector<uint8_t> referenced(A, 0);
  for (int32_t r = 0; r < R; ++r)
    if (b->agent[r] >= 0) referenced[b->agent[r]] = 1;
  int64_t need = 0;
  for (int32_t a = 0; a < A; ++a)
    if (referenced[a]) need += pages_for(pt->prefix_len[a]);
  for (int32_t r = 0; r < R; ++r) need += pages_for(b->suffix_len[r]);
  if (need > pool->num_pages)
    return fail(PFX_ENOMEM, "pfx_plan_create: batch needs %lld pages (prefixes once + suffixes), pool has %d",
                (long long)need, pool->num_pages);

  // ---- page ids: in range and owned exactly once ----
  std::vector<uint64_t> owner((size_t(pool->num_pages) + 63) / 64, 0);  // one bit per page
  auto claim = [&](int32_t id, const char* what, int32_t who) -> int {
    if (id < 0 || id >= pool->num_pages)
      return fail(PFX_ERANGE, "pfx_plan_create: %s %d uses page %d outside [0, %d)", what, who, id, pool->num_pages);
    const uint64_t bit = uint64_t(1) << (id & 63);
    if (owner[id >> 6] & bit) return fail(PFX_EINVAL, "pfx_plan_create: page %d is used twice (%s %d)", id, what, who);
    owner[id >> 6] |= bit;
    return PFX_OK;
  };
  for (int32_t a = 0; a < A; ++a) {
    if (!referenced[a]) continue;
    for (int32_t i = pt->page_indptr[a]; i < pt->page_indptr[a + 1]; ++i)
      if ((rc = claim(pt->page_ids[i], "agent", a))) return rc;
  }
  for (int32_t r = 0; r < R; ++r)
    for (int32_t i = b->suffix_indptr[r]; i < b->suffix_indptr[r + 1]; ++i)
      if ((rc = claim(b->suffix_page_ids[i], "request", r))) return rc;

  // ---- build ----
  pfx_plan* p = new (std::nothrow) pfx_plan;
  if (!p) return fail(PFX_ENOMEM, "pfx_plan_create: host allocation failed");
  p->num_pages = pool->num_pages;
  p->hkv = hkv;
  p->d = pool->head_dim;
  p->hq = hq;
  p->group = G;
  p->mode = mode;
  p->decode_workers = p_workers;
  p->decode_engine = engine;
  p->num_reqs = R;
  p->num_tokens = static_cast<int32_t>(total_tokens);
  p->pages_needed = static_cast<int32_t>(need);

  std::vector<int32_t> prefix_off(A, -1), suffix_off(R, 0);
  for (int32_t a = 0; a < A; ++a) {
    if (!referenced[a]) continue;
    prefix_off[a] = static_cast<int32_t>(p->page_list.size());
    p->page_list.insert(p->page_list.end(), pt->page_ids + pt->page_indptr[a], pt->page_ids + pt->page_indptr[a + 1]);
  }
  for (int32_t r = 0; r < R; ++r) {
    suffix_off[r] = static_cast<int32_t>(p->page_list.size());
    p->page_list.insert(p->page_list.end(), b->suffix_page_ids + b->suffix_indptr[r],
                        b->suffix_page_ids + b->suffix_indptr[r + 1]);
  }
  p->tok_req.resize(total_tokens);
  p->tok_slot.resize(total_tokens);
  p->req.resize(R);
  for (int32_t r = 0; r < R; ++r) {
    const int32_t q0 = b->q_indptr[r], n = b->q_indptr[r + 1] - q0, L = b->suffix_len[r];
    p->req[r] = ReqInfo{q0, n};
    for (int32_t i = 0; i < n; ++i) {
      int32_t pos = L - n + i;
      int32_t page = b->suffix_page_ids[b->suffix_indptr[r] + pos / PFX_PAGE_SIZE];
      p->tok_req[q0 + i] = r;
      p->tok_slot[q0 + i] = page * PFX_PAGE_SIZE + pos % PFX_PAGE_SIZE;
    }
  }

  auto is_decode_class = [&](int32_t r) {
    int32_t n = p->req[r].n;
    return n >= 1 && n * G <= kTileCols;
  };
  auto blocks_for = [&](int32_t tokens) { return (tokens * G + kTileCols - 1) / kTileCols; };

  // ---- decode items (Sec. 3): each agent's prefix once per block of its
  // decode rows and KV head, then each request's own suffix per KV head ----
  struct DItem {
    int32_t kind, h, keys, page_off, causal_base;
    int32_t row_first, rows;  // tokens drow_tok[row_first .. + rows)
    int64_t step_first;
    int32_t npieces;
    int32_t wide;             // a prefix item of up to 128 columns, run as wide blocks (32 columns per wave)
  };
  std::vector<DItem> dit;
  std::vector<int32_t> drow_tok;
  std::vector<int32_t> pf_item(size_t(R) * hkv, -1), sf_item(size_t(R) * hkv, -1);
  for (int32_t a = 0; a < A; ++a) {
    if (!referenced[a] || pt->prefix_len[a] == 0) continue;
    std::vector<int32_t> members;
    int64_t agent_cols = 0;
    for (int32_t r = 0; r < R; ++r)
      if (b->agent[r] == a && is_decode_class(r)) {
        members.push_back(r);
        agent_cols += int64_t(p->req[r].n) * G;
      }
    // An agent with more decode columns per KV head than one 64-column
    // piece holds reads each prefix step for up to 128 columns at once
    // (wide blocks): half the stages, each with twice the products.
    const int32_t wide = engine == PFX_DECODE_MFMA && agent_cols > kDecodeTileCols;
    const int32_t block_cols = wide ? kExtendTileCols : kDecodeTileCols;
    size_t i = 0;
    while (i < members.size()) {
      // A block of rows whose columns (rows x G) fit one item.
      const int32_t first = static_cast<int32_t>(drow_tok.size());
      int32_t cols = 0;
      std::vector<int32_t> in_block;
      while (i < members.size() && cols + p->req[members[i]].n * G <= block_cols) {
        const int32_t r = members[i++];
        for (int32_t t = 0; t < p->req[r].n; ++t) drow_tok.push_back(p->req[r].q_start + t);
        cols += p->req[r].n * G;
        in_block.push_back(r);
      }
      const int32_t rows = static_cast<int32_t>(drow_tok.size()) - first;
      for (int32_t h = 0; h < hkv; ++h) {
        for (int32_t r : in_block) pf_item[size_t(r) * hkv + h] = static_cast<int32_t>(dit.size());
        dit.push_back(DItem{kPrefixItem, h, pt->prefix_len[a], prefix_off[a], 0, first, rows, 0, 0, wide});
        ++p->n_prefix_items;
      }
    }
  }
  for (int32_t r = 0; r < R; ++r) {
    if (!is_decode_class(r)) continue;
    const ReqInfo ri = p->req[r];
    const int32_t L = b->suffix_len[r];  // >= n >= 1: the suffix holds the new tokens
    const int32_t first = static_cast<int32_t>(drow_tok.size());
    for (int32_t t = 0; t < ri.n; ++t) drow_tok.push_back(ri.q_start + t);
    for (int32_t h = 0; h < hkv; ++h) {
      sf_item[size_t(r) * hkv + h] = static_cast<int32_t>(dit.size());
      dit.push_back(DItem{kSuffixItem, h, L, suffix_off[r], L - ri.n - ri.q_start, first, ri.n, 0, 0, 0});
      ++p->n_suffix_items;
    }
  }

  // ---- decode pieces: each item's 32-key steps (two 16-key pages of one
  // KV head) cut into runs of at most kPieceSteps, as even as possible ----
  auto page_blk = [&](const DItem& x, int32_t pg) { return p->page_list[x.page_off + pg] * hkv + x.h; };
  // A piece is described by its item, its index and its step range here; the
  // full records are written once, in launch order, further down.
  struct Piece {
    int32_t item, piece, s0, s1;
  };
  std::vector<Piece> pcs;
  if (piece_steps == 0) {
    int64_t steps = 0;
    for (const DItem& x : dit) steps += (x.keys + kStepKeys - 1) / kStepKeys;
    piece_steps = steps >= kLongPiecesFrom ? kLongPieceSteps : kDefaultPieceSteps;
  }
  {
    size_t total = 0;
    for (const DItem& x : dit) {
      const int32_t ns = (x.keys + kStepKeys - 1) / kStepKeys;
      total += size_t((ns + piece_steps - 1) / piece_steps);
    }
    pcs.reserve(total);
  }
  for (size_t xi = 0; xi < dit.size(); ++xi) {
    const int32_t ns = (dit[xi].keys + kStepKeys - 1) / kStepKeys;
    const int32_t np = (ns + piece_steps - 1) / piece_steps;
    p->num_decode_steps += ns;
    for (int32_t k = 0; k < np; ++k)
      pcs.push_back(Piece{static_cast<int32_t>(xi), k, int32_t(int64_t(k) * ns / np), int32_t(int64_t(k + 1) * ns / np)});
    dit[xi].npieces = np;
  }

  // ---- partial slots: a decode row of KV head h is seen by the pieces of
  // its prefix item (slots 0 ..) and then of its suffix item; every piece
  // leaves its unnormalised state in a slot and the log-sum-exp merge
  // combines them into the row (a lone piece is just normalised) ----
  // A decode request's rows are consecutive in the merge list, from
  // req_mrow[r]; merge_head[row * Hkv + h] holds their first slot and count.
  std::vector<int32_t> np_prefix(size_t(R) * hkv, 0), np_total(size_t(R) * hkv, 0), req_mrow(R, -1);
  int64_t part_units = 0;
  for (int32_t r = 0; r < R; ++r) {
    if (!is_decode_class(r)) continue;
    bool any = false;
    for (int32_t h = 0; h < hkv; ++h) {
      const size_t rh = size_t(r) * hkv + h;
      np_prefix[rh] = pf_item[rh] >= 0 ? dit[pf_item[rh]].npieces : 0;
      np_total[rh] = np_prefix[rh] + dit[sf_item[rh]].npieces;
      any |= np_total[rh] >= 1;
    }
    if (!any) continue;
    req_mrow[r] = static_cast<int32_t>(p->merge_tok.size());
    for (int32_t t = 0; t < p->req[r].n; ++t) {
      const int32_t tok = p->req[r].q_start + t;
      p->merge_tok.push_back(tok);
      for (int32_t h = 0; h < hkv; ++h) {
        const int32_t np = np_total[size_t(r) * hkv + h];
        if (np >= 1) {
          p->merge_head.push_back(MergeHead{static_cast<int32_t>(part_units), np});
          part_units += np;
        } else {
          p->merge_head.push_back(MergeHead{0, 0});
        }
      }
    }
  }
  if (part_units * G > (int64_t(1) << 31) / std::max(1, p->d))
    return delete p, fail(PFX_ERANGE, "pfx_plan_create: too many partial rows");
  p->num_part_rows = part_units * G;
  // When every (merge row, KV head) has the same number of parts P, its
  // slots start at (row * Hkv + h) * P, and the merge launch computes that
  // instead of loading merge_head (one dependent round trip less).
  p->merge_parts = 0;
  if (!p->merge_head.empty()) {
    const int32_t P = p->merge_head[0].nparts;
    bool uniform = P >= 1;
    for (size_t i = 0; uniform && i < p->merge_head.size(); ++i)
      uniform = p->merge_head[i].nparts == P && int64_t(p->merge_head[i].base) == int64_t(i) * P;
    if (uniform) p->merge_parts = P;
  }
  // Merge row m is decode token m (a batch of decode rows only, in order):
  // the merge launch then needs no merge_tok load either.
  p->merge_tok_is_row = 1;
  for (size_t m = 0; p->merge_tok_is_row && m < p->merge_tok.size(); ++m)
    p->merge_tok_is_row = p->merge_tok[m] == int32_t(m);

  // Longest first: a prefix step multiplies 64 query columns, a suffix step
  // at most 16, so prefix steps weigh a little more (a wide prefix step,
  // 128 columns, twice as much); every piece also has a stage for its query
  // rows.
  const size_t npcs = pcs.size();
  auto is_prefix = [&](int32_t k) { return dit[pcs[k].item].kind == kPrefixItem; };
  auto is_wide = [&](int32_t k) { return dit[pcs[k].item].wide != 0; };
  std::vector<int32_t> pcost(npcs), rank(npcs);
  for (size_t k = 0; k < npcs; ++k) {
    const int32_t w = is_wide(int32_t(k)) ? 22 : is_prefix(int32_t(k)) ? 11 : 10;
    pcost[k] = w * (pcs[k].s1 - pcs[k].s0) + 10;
    rank[k] = static_cast<int32_t>(k);
  }
  std::stable_sort(rank.begin(), rank.end(), [&](int32_t x, int32_t y) { return pcost[x] > pcost[y]; });

  // The column blocks of one prefix chunk (one KV head, the same steps of an
  // agent's prefix, different decode rows) read the same K/V.  Pieces are
  // dealt to workgroup p mod S in even rounds and S - 1 - p mod S in odd
  // ones, and the dispatcher hands workgroups to the 8 XCDs in turn, so
  // positions eight apart in one round run on one XCD.  Within each run of
  // equal-cost prefix pieces, chunks are taken eight at a time and block j
  // of the c-th is placed at 8 j + c: a chunk's blocks then run side by side
  // behind one L2 and read it from HBM about once.  Only the order changes
  // (every piece keeps its partial slot), so results do not.
  std::vector<int32_t> order;
  order.reserve(npcs);
  {
    size_t i = 0;
    while (i < npcs) {
      const int32_t cost = pcost[rank[i]];
      const bool prefix = is_prefix(rank[i]);
      size_t j = i;
      while (j < npcs && pcost[rank[j]] == cost && is_prefix(rank[j]) == prefix) ++j;
      if (!prefix) {
        order.insert(order.end(), rank.begin() + i, rank.begin() + j);
        i = j;
        continue;
      }
      // A chunk is named by the page block of its first step.
      std::vector<std::vector<int32_t>> chunks;
      std::unordered_map<int32_t, size_t> chunk_of;
      for (size_t k = i; k < j; ++k) {
        const Piece& pc = pcs[rank[k]];
        auto ins = chunk_of.emplace(page_blk(dit[pc.item], 2 * pc.s0), chunks.size());
        if (ins.second) chunks.emplace_back();
        chunks[ins.first->second].push_back(rank[k]);
      }
      // Chunks with the same number of blocks go together, so a group of
      // eight has complete rounds: its first `common` blocks are laid out
      // eight apart, and blocks past a shorter chunk's end go to the end of
      // the run (placed there, they would shift every later position).
      std::stable_sort(chunks.begin(), chunks.end(),
                       [](const std::vector<int32_t>& x, const std::vector<int32_t>& y) { return x.size() > y.size(); });
      std::vector<int32_t> leftover;
      for (size_t g = 0; g < chunks.size(); g += 8) {
        const size_t g1 = std::min(chunks.size(), g + 8);
        size_t common = chunks[g].size();
        for (size_t c = g; c < g1; ++c) common = std::min(common, chunks[c].size());
        for (size_t bj = 0; bj < common; ++bj)
          for (size_t c = g; c < g1; ++c) order.push_back(chunks[c][bj]);
        for (size_t c = g; c < g1; ++c)
          for (size_t bj = common; bj < chunks[c].size(); ++bj) leftover.push_back(chunks[c][bj]);
      }
      order.insert(order.end(), leftover.begin(), leftover.end());
      i = j;
    }
  }

  // Wide pieces run as blocks of the attention launch ahead of the decode
  // pieces (in this order, so a chunk's blocks still sit eight apart); the
  // others are decode pieces.
  std::vector<int32_t> wide_order, seg_order;
  for (int32_t k : order) (is_wide(k) ? wide_order : seg_order).push_back(k);
  const size_t nsegs = seg_order.size();
  if (nsegs > size_t(INT32_MAX) || wide_order.size() > size_t(INT32_MAX))
    return delete p, fail(PFX_ERANGE, "pfx_plan_create: too many decode pieces");

  // ---- extend blocks (Sec. 3): up to 128 query columns of one request,
  // over the whole prefix (no mask) then the suffix (causal), written
  // directly ----
  // A block of rows of one request, before it is expanded over the KV heads.
  struct XBlock {
    int32_t r, i0, i1, rbeg;
    int64_t cost;  // keys it streams: the whole prefix and the suffix up to its last row
  };
  std::vector<XBlock> xbs;
  p->row_tok.reserve(total_tokens);
  for (int32_t r = 0; r < R; ++r) {
    const ReqInfo ri = p->req[r];
    if (ri.n == 0 || is_decode_class(r)) continue;
    const int32_t a = b->agent[r];
    const int32_t P = a >= 0 ? pt->prefix_len[a] : 0;
    const int32_t L = b->suffix_len[r];
    const int32_t per = kExtendTileCols / G;
    for (int32_t i0 = 0; i0 < ri.n; i0 += per) {
      const int32_t i1 = std::min(ri.n, i0 + per);
      const int32_t rbeg = static_cast<int32_t>(p->row_tok.size());
      for (int32_t i = i0; i < i1; ++i) p->row_tok.push_back(ri.q_start + i);
      xbs.push_back(XBlock{r, i0, i1, rbeg, int64_t(P) + (L - ri.n + i1)});
    }
  }
  // Rows of the wide prefix blocks: their tokens and the partial row each
  // (token, slot) leaves its state in (extend rows have no partial row).
  p->row_out.assign(p->row_tok.size(), -1);
  std::vector<int32_t> wide_rbeg(wide_order.size());
  for (size_t w = 0; w < wide_order.size(); ++w) {
    const Piece& pc = pcs[wide_order[w]];
    const DItem& x = dit[pc.item];
    wide_rbeg[w] = static_cast<int32_t>(p->row_tok.size());
    for (int32_t j = 0; j < x.rows; ++j) {
      const int32_t tok = drow_tok[x.row_first + j];
      const int32_t r = p->tok_req[tok];
      const size_t mrow = size_t(req_mrow[r]) + (tok - p->req[r].q_start);
      p->row_tok.push_back(tok);
      p->row_out.push_back((p->merge_head[mrow * hkv + x.h].base + pc.piece) * G);
    }
  }

  // Blocks of one agent together, longest key ranges first within it.  The
  // KV heads of one block stay together, in order, and the dispatcher deals
  // workgroups to the 8 XCDs in turn, so with 8 KV heads an XCD runs one
  // head: grouped by agent, the blocks it runs at a time read one prefix,
  // about the same keys at about the same time, through its L2 (ordered by
  // length alone, they read every agent's prefix at once).  The launch still
  // ends on the shortest blocks of the last agent.
  std::vector<int32_t> xrank(xbs.size());
  for (size_t k = 0; k < xbs.size(); ++k) xrank[k] = static_cast<int32_t>(k);
  std::stable_sort(xrank.begin(), xrank.end(), [&](int32_t x, int32_t y) {
    const int32_t ax = b->agent[xbs[x].r], ay = b->agent[xbs[y].r];
    if (ax != ay) return ax > ay;  // requests without a prefix (-1) last
    return xbs[x].cost > xbs[y].cost;
  });
  const size_t nitems = xbs.size() * size_t(hkv);
  if (nitems + wide_order.size() > size_t(INT32_MAX))
    return delete p, fail(PFX_ERANGE, "pfx_plan_create: too many extend blocks");
  p->n_extend_items = static_cast<int32_t>(nitems);
  p->num_wide = static_cast<int32_t>(wide_order.size());

  // ---- workspace layout ----
  size_t off = 0;
  p->off_items = off;      off = align256(off + (nitems + wide_order.size()) * sizeof(Item));
  p->off_row_tok = off;    off = align256(off + p->row_tok.size() * 4);
  p->off_row_out = off;    off = align256(off + p->row_out.size() * 4);
  p->off_page_list = off;  off = align256(off + p->page_list.size() * 4);
  p->off_tok_slot = off;   off = align256(off + p->tok_slot.size() * 4);
  p->off_segs = off;       off = align256(off + nsegs * sizeof(Seg));
  p->off_merge_tok = off;  off = align256(off + p->merge_tok.size() * 4);
  p->off_merge_head = off; off = align256(off + p->merge_head.size() * sizeof(MergeHead));
  p->blob_bytes = off;
  p->off_opart = off;      off = align256(off + size_t(p->num_part_rows) * p->d * 2);
  p->off_lpart = off;      off = align256(off + size_t(p->num_part_rows) * 8);
  p->total_bytes = std::max<size_t>(off, 256);

  p->num_items = static_cast<int32_t>(nitems);
  p->num_segs = static_cast<int32_t>(nsegs);

  // The host image: the last destroyed plan's buffer is reused when it is
  // large enough (a serving loop builds a plan every step, and fresh pages
  // of a few hundred KiB cost more to fault in than to fill).
  // Every byte of the image is written once: each section by its copy or
  // its records below, the alignment gaps after the sections here (the
  // reused buffer may still hold the last plan's bytes).
  p->blob.swap(spare_blob());
  p->blob.resize(p->blob_bytes);
  {
    const size_t sect[][2] = {
        {p->off_items, (nitems + wide_order.size()) * sizeof(Item)},
        {p->off_row_tok, p->row_tok.size() * 4},
        {p->off_row_out, p->row_out.size() * 4},
        {p->off_page_list, p->page_list.size() * 4},
        {p->off_tok_slot, p->tok_slot.size() * 4},
        {p->off_segs, nsegs * sizeof(Seg)},
        {p->off_merge_tok, p->merge_tok.size() * 4},
        {p->off_merge_head, p->merge_head.size() * sizeof(MergeHead)},
    };
    const size_t ns = sizeof(sect) / sizeof(sect[0]);
    for (size_t i = 0; i < ns; ++i) {
      const size_t end = sect[i][0] + sect[i][1], next = i + 1 < ns ? sect[i + 1][0] : p->blob_bytes;
      if (next > end) std::memset(p->blob.data() + end, 0, next - end);
    }
  }
  auto put = [&](size_t at, const void* src, size_t bytes) {
    if (bytes) std::memcpy(p->blob.data() + at, src, bytes);
  };
  put(p->off_row_tok, p->row_tok.data(), p->row_tok.size() * 4);
  put(p->off_row_out, p->row_out.data(), p->row_out.size() * 4);
  put(p->off_page_list, p->page_list.data(), p->page_list.size() * 4);
  put(p->off_tok_slot, p->tok_slot.data(), p->tok_slot.size() * 4);
  put(p->off_merge_tok, p->merge_tok.data(), p->merge_tok.size() * 4);
  put(p->off_merge_head, p->merge_head.data(), p->merge_head.size() * sizeof(MergeHead));

  // The extend block records, in launch order: each block's leading page
  // ids and first token are filled in here.
  Item* items = reinterpret_cast<Item*>(p->blob.data() + p->off_items);
  size_t nit = 0;
  for (int32_t xi : xrank) {
    const XBlock& xb = xbs[xi];
    const ReqInfo ri = p->req[xb.r];
    const int32_t a = b->agent[xb.r];
    const int32_t P = a >= 0 ? pt->prefix_len[a] : 0;
    const int32_t L = b->suffix_len[xb.r];
    Item it{};  // the same for every KV head but the head itself
    it.row_begin = xb.rbeg;
    it.row_count = xb.i1 - xb.i0;
    it.nblk = blocks_for(xb.i1 - xb.i0);
    it.s0_page_off = P > 0 ? prefix_off[a] : 0;
    it.s0_kbeg = 0;
    it.s0_kend = P;
    it.s1_page_off = suffix_off[xb.r];
    it.s1_kbeg = 0;
    it.s1_kend = L - ri.n + xb.i1;
    it.causal_base = L - ri.n - ri.q_start;
    it.out_slot = -1;
    it.kind = kExtendItem;
    it.req = xb.r;
    int32_t k = 0;
    for (int32_t pg = it.s0_kbeg >> 4; it.s0_kend > it.s0_kbeg && pg < (it.s0_kend + 15) >> 4 && k < kItemPages; ++pg)
      it.first_pages[k++] = p->page_list[it.s0_page_off + pg];
    for (int32_t pg = it.s1_kbeg >> 4; it.s1_kend > it.s1_kbeg && pg < (it.s1_kend + 15) >> 4 && k < kItemPages; ++pg)
      it.first_pages[k++] = p->page_list[it.s1_page_off + pg];
    it.tok0 = p->row_tok[it.row_begin];
    for (int32_t h = 0; h < hkv; ++h) {
      it.kv_head = h;
      new (items + nit++) Item(it);
    }
  }

  // The wide prefix blocks, after the extend blocks: one piece of the
  // agent's prefix (segment 0) against the block's decode rows, leaving
  // partial states.
  for (size_t w = 0; w < wide_order.size(); ++w) {
    const Piece& pc = pcs[wide_order[w]];
    const DItem& x = dit[pc.item];
    Item it{};
    it.kv_head = x.h;
    it.row_begin = wide_rbeg[w];
    it.row_count = x.rows;
    it.nblk = blocks_for(x.rows);
    it.s0_page_off = x.page_off;
    it.s0_kbeg = pc.s0 * kStepKeys;
    it.s0_kend = std::min(pc.s1 * kStepKeys, x.keys);
    it.out_slot = pc.piece;
    it.kind = kPrefixItem;
    it.req = -1;
    it.tok0 = -1;
    for (int32_t k = 0, pg = it.s0_kbeg >> 4; pg < (it.s0_kend + 15) >> 4 && k < kItemPages; ++pg)
      it.first_pages[k++] = p->page_list[it.s0_page_off + pg];
    new (items + nit++) Item(it);
  }

  // The piece records, in launch order.
  Seg* segs = reinterpret_cast<Seg*>(p->blob.data() + p->off_segs);
  for (size_t k = 0; k < nsegs; ++k) {
    const Piece& pc = pcs[seg_order[k]];
    const DItem& x = dit[pc.item];
    const int32_t npages = static_cast<int32_t>(pages_for(x.keys));
    Seg& sg = *new (segs + k) Seg{};
    sg.h.kind = x.kind;
    sg.h.kv_head = x.h;
    sg.h.ncols = x.rows * G;
    sg.h.nsteps = pc.s1 - pc.s0;
    sg.h.k0 = pc.s0 * kStepKeys;
    sg.h.kend = x.keys;
    sg.h.causal_base = x.causal_base;
    sg.h.causal = x.kind == kSuffixItem && x.rows > 1;
    sg.h.item = pc.item;
    sg.h.piece = pc.piece;
    for (int32_t i = pc.s0; i < pc.s1; ++i) {
      const int32_t pg0 = 2 * i, pg1 = 2 * i + 1 < npages ? 2 * i + 1 : 2 * i;  // a missing page repeats (masked)
      sg.steps[2 * (i - pc.s0)] = page_blk(x, pg0);
      sg.steps[2 * (i - pc.s0) + 1] = page_blk(x, pg1);
    }
    for (int32_t j = 0; j < x.rows; ++j) {
      const int32_t tok = drow_tok[x.row_first + j];
      const int32_t r = p->tok_req[tok];
      const size_t rh = size_t(r) * hkv + x.h;
      sg.tok[j] = tok;
      const int32_t slot = (x.kind == kPrefixItem ? 0 : np_prefix[rh]) + pc.piece;
      sg.h.slot = slot;  // the same for every row of the piece
      const size_t mrow = size_t(req_mrow[r]) + (tok - p->req[r].q_start);
      sg.out[j] = (p->merge_head[mrow * hkv + x.h].base + slot) * G;
    }
  }

  *out = p;
  return PFX_OK;
}

extern "C" int pfx_plan_workspace_bytes(const pfx_plan* p, size_t* bytes) {
  if (!p || !bytes) return fail(PFX_EINVAL, "pfx_plan_workspace_bytes: NULL argument");
  *bytes = p->total_bytes;
  return PFX_OK;
}

extern "C" int pfx_plan_get_stats(const pfx_plan* p, pfx_plan_stats* s) {
  if (!p || !s) return fail(PFX_EINVAL, "pfx_plan_get_stats: NULL argument");
  s->num_requests = p->num_reqs;
  s->num_tokens = p->num_tokens;
  s->num_items = p->n_prefix_items + p->n_suffix_items + p->n_extend_items;
  s->num_prefix_items = p->n_prefix_items;
  s->num_suffix_items = p->n_suffix_items;
  s->num_extend_items = p->n_extend_items;
  s->num_partial_rows = static_cast<int32_t>(p->num_part_rows);
  s->pages_needed = p->pages_needed;
  s->num_decode_steps = static_cast<int32_t>(p->num_decode_steps);
  s->num_decode_pieces = p->num_segs;
  s->num_wide_blocks = p->num_wide;
  s->reserved = 0;
  s->workspace_bytes = static_cast<int64_t>(p->total_bytes);
  return PFX_OK;
}

extern "C" int pfx_plan_export(const pfx_plan* p, int32_t which, int32_t* out, int64_t cap, int64_t* count) {
  if (!p || !count) return fail(PFX_EINVAL, "pfx_plan_export: NULL argument");
  const int32_t* src = nullptr;
  int64_t n = 0;
  switch (which) {
    case 0: src = reinterpret_cast<const int32_t*>(p->host_items()); n = int64_t(p->num_items + p->num_wide) * 32; break;
    case 1: src = p->row_tok.data(); n = int64_t(p->row_tok.size()); break;
    case 8: src = p->row_out.data(); n = int64_t(p->row_out.size()); break;
    case 2: src = p->page_list.data(); n = int64_t(p->page_list.size()); break;
    case 3: src = reinterpret_cast<const int32_t*>(p->host_segs()); n = int64_t(p->num_segs) * 272; break;
    case 6: src = p->merge_tok.data(); n = int64_t(p->merge_tok.size()); break;
    case 7: src = reinterpret_cast<const int32_t*>(p->merge_head.data()); n = int64_t(p->merge_head.size()) * 2; break;
    default: return fail(PFX_EINVAL, "pfx_plan_export: which = %d", which);
  }
  *count = n;
  if (cap > 0 && !out) return fail(PFX_EINVAL, "pfx_plan_export: out is NULL");
  int64_t m = std::min(n, std::max<int64_t>(cap, 0));
  if (m) std::memcpy(out, src, size_t(m) * 4);
  return PFX_OK;
}

extern "C" void pfx_plan_destroy(pfx_plan* p) {
  if (!p) return;
  std::vector<unsigned char>& spare = pfx::spare_blob();
  if (p->blob.capacity() > spare.capacity()) spare.swap(p->blob);
  delete p;
}

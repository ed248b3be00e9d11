// Host-only driver of the plan builder and the page allocator, built with
// the address and undefined-behaviour sanitizers (no HIP: pfx_plan.cpp is
// compiled on its own).  Reads cases from a text file, one per block:
//   num_pages hkv d hq mode piece_steps decode_workers
//   A  prefix_len[A]  page_indptr[A+1]  page_ids[page_indptr[A]]
//   R  agent[R]  suffix_indptr[R+1]  suffix_page_ids[suffix_indptr[R]]  suffix_len[R]  q_indptr[R+1]
// and prints, per case, the status and the plan's counts (or the error
// text), then exercises the allocator.  Every array is read into a vector
// of exactly its length, so a read past its end is caught.
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/pfx_attn.h"

static bool read_vec(FILE* f, std::vector<int32_t>& v, long n) {
  v.assign(n, 0);
  for (long i = 0; i < n; ++i)
    if (fscanf(f, "%d", &v[i]) != 1) return false;
  return true;
}

int main(int argc, char** argv) {
  if (argc != 2) return 2;
  FILE* f = fopen(argv[1], "r");
  if (!f) return 2;
  int cases = 0;
  pfx_pool pool;
  int hq, mode, piece_steps, workers;
  while (fscanf(f, "%d %d %d %d %d %d %d", &pool.num_pages, &pool.num_kv_heads, &pool.head_dim, &hq, &mode,
                &piece_steps, &workers) == 7) {
    pool.page_size = PFX_PAGE_SIZE;
    pool.k_pages = pool.v_pages = nullptr;
    int A = 0, R = 0;
    std::vector<int32_t> plen, pind, pids, agent, sind, sids, slen, qind;
    if (fscanf(f, "%d", &A) != 1 || !read_vec(f, plen, A) || !read_vec(f, pind, A + 1) ||
        !read_vec(f, pids, A ? pind[A] : 0))
      return 3;
    if (fscanf(f, "%d", &R) != 1 || !read_vec(f, agent, R) || !read_vec(f, sind, R + 1) ||
        !read_vec(f, sids, R ? sind[R] : 0) || !read_vec(f, slen, R) || !read_vec(f, qind, R + 1))
      return 3;
    pfx_prefix_table pt = {A, pind.data(), pids.data(), plen.data()};
    pfx_batch b = {R, agent.data(), sind.data(), sids.data(), slen.data(), qind.data()};
    pfx_plan_opts opts;
    memset(&opts, 0, sizeof(opts));
    opts.piece_steps = piece_steps;
    opts.decode_workers = workers;
    pfx_plan* p = nullptr;
    int rc = pfx_plan_create(&pool, &pt, &b, hq, mode, &opts, &p);
    if (rc != PFX_OK) {
      printf("case %d rc %d %s\n", cases, rc, pfx_last_error());
    } else {
      pfx_plan_stats s;
      pfx_plan_get_stats(p, &s);
      size_t ws = 0;
      pfx_plan_workspace_bytes(p, &ws);
      int64_t total = 0;
      for (int which : {0, 1, 2, 3, 6, 7}) {
        int64_t n = 0;
        pfx_plan_export(p, which, nullptr, 0, &n);
        std::vector<int32_t> out(n);
        pfx_plan_export(p, which, out.data(), n, &n);
        for (int32_t x : out) total += x;
      }
      printf("case %d rc 0 tokens %d items %d pieces %d partial %d pages %d ws %zu sum %lld\n", cases, s.num_tokens,
             s.num_items, s.num_decode_pieces, s.num_partial_rows, s.pages_needed, ws, (long long)total);
      pfx_plan_destroy(p);
    }
    ++cases;
  }
  fclose(f);
  // The allocator: hand out, free, fail cleanly.
  pfx_alloc* a = nullptr;
  if (pfx_alloc_create(100, &a) != PFX_OK) return 4;
  std::vector<int32_t> ids(60);
  if (pfx_alloc_pages(a, 60, ids.data()) != PFX_OK) return 4;
  if (pfx_alloc_pages(a, 41, ids.data()) != PFX_ENOMEM) return 4;
  if (pfx_free_pages(a, ids.data(), 30) != PFX_OK) return 4;
  if (pfx_free_pages(a, ids.data(), 1) != PFX_EINVAL) return 4;   // freed twice
  int32_t n = 0;
  pfx_alloc_num_free(a, &n);
  pfx_alloc_destroy(a);
  printf("allocator free %d\n", n);
  return n == 70 ? 0 : 4;
}

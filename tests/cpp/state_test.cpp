// Host-only checks of the context bookkeeping (csrc/host/state.h), built with
// g++ and sanitizers by tests/test_abi_cpu.py.
#include <stdio.h>
#include <stdlib.h>

#include "state.h"

using namespace ams;

static int failures = 0;
#define EXPECT(c)                                                  \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "%s:%d: EXPECT(%s) failed\n", __FILE__, __LINE__, #c); \
      ++failures;                                                  \
    }                                                              \
  } while (0)

static void test_book() {
  RowBook b;
  b.init(3, 128);
  std::string e;
  int32_t nl[3] = {0, 0, 0};
  EXPECT(b.check_step(nl, 7, e) == S_ESTATE);  // never built
  int32_t bad[3] = {10, 0, 5};
  EXPECT(b.check_build(bad, e) == S_EINVAL);
  int32_t big[3] = {10, 129, 5};
  EXPECT(b.check_build(big, e) == S_ECAPACITY);
  int32_t lens[3] = {100, 1, 128};
  EXPECT(b.check_build(lens, e) == S_OK);
  b.commit_build(lens);
  EXPECT(b.state == READY);
  EXPECT(b.check_step(nullptr, 1, e) == S_OK);       // 128 + 0 + 1 - 1 = 128 fits
  EXPECT(b.check_step(nullptr, 2, e) == S_ECAPACITY);
  int32_t l2[3] = {90, 1, 100};
  b.commit_build(l2);
  int32_t n1[3] = {28, 0, 0};
  EXPECT(b.check_step(n1, 11, e) == S_OK);          // 90 + 28 + 11 - 1 = 128: exact fit
  EXPECT(b.check_step(n1, 12, e) == S_ECAPACITY);
  int32_t neg[3] = {0, -1, 0};
  EXPECT(b.check_step(neg, 1, e) == S_EINVAL);
  EXPECT(b.check_step(nullptr, 0, e) == S_EINVAL);
  b.commit_new(n1);
  EXPECT(b.len[0] == 118 && b.len[1] == 1 && b.len[2] == 100);
  b.invalidate();
  EXPECT(b.state == INVALID && b.len[0] == 0 && b.len[2] == 0);
  EXPECT(b.check_step(nullptr, 1, e) == S_ESTATE);
  b.commit_build(l2);
  EXPECT(b.state == READY && b.len[2] == 100);
}

// The persistent decode reports a barrier wait that gave up through a status
// word; the next call on the context maps it to S_EHIP and an INVALID context.
static void test_async_error() {
  RowBook b;
  b.init(2, 64);
  std::string e;
  int32_t lens[2] = {10, 20};
  b.commit_build(lens);
  EXPECT(b.absorb_async_error(0u, e) == S_OK);  // clean word: nothing changes
  EXPECT(b.state == READY && b.len[1] == 20);
  EXPECT(b.absorb_async_error(1u, e) == S_EHIP);
  EXPECT(b.state == INVALID && b.len[0] == 0 && b.len[1] == 0);
  EXPECT(!e.empty());
  EXPECT(b.check_step(nullptr, 1, e) == S_ESTATE);  // stepping now needs a rebuild
  b.commit_build(lens);
  EXPECT(b.state == READY && b.check_step(nullptr, 1, e) == S_OK);
}

// Row-level invalidate / rebuild inside a live batch, and append-only commits.
static void test_rows() {
  RowBook b;
  b.init(4, 128);
  std::string e;
  int32_t r1[1] = {2}, l1[1] = {50};
  EXPECT(b.check_build_rows(r1, 1, l1, e) == S_OK);
  b.commit_build_rows(r1, 1, l1);
  EXPECT(b.state == INVALID);  // rows 0, 1, 3 never built: not steppable
  EXPECT(b.check_step(nullptr, 1, e) == S_ESTATE);
  int32_t r3[3] = {0, 1, 3}, l3[3] = {10, 20, 30};
  b.commit_build_rows(r3, 3, l3);
  EXPECT(b.state == READY && b.len[2] == 50 && b.len[3] == 30);
  int32_t unsorted[2] = {3, 1}, dup[2] = {1, 1}, oob[1] = {4};
  EXPECT(b.check_rows(unsorted, 2, e) == S_EINVAL);
  EXPECT(b.check_rows(dup, 2, e) == S_EINVAL);
  EXPECT(b.check_rows(oob, 1, e) == S_EINVAL);
  EXPECT(b.check_rows(r1, 0, e) == S_EINVAL);
  int32_t toolong[1] = {129}, zero[1] = {0};
  EXPECT(b.check_build_rows(r1, 1, toolong, e) == S_ECAPACITY);
  EXPECT(b.check_build_rows(r1, 1, zero, e) == S_EINVAL);
  // one robot's exception: row 1 discarded, the others keep their lengths
  int32_t one[1] = {1};
  b.invalidate_rows(one, 1);
  EXPECT(b.state == INVALID && b.len[1] == 0 && b.len[0] == 10 && b.len[3] == 30);
  int32_t nl[4] = {1, 1, 1, 1};
  EXPECT(b.check_append(nl, e) == S_ESTATE);
  EXPECT(b.check_step(nullptr, 1, e) == S_ESTATE);
  int32_t l9[1] = {9};
  b.commit_build_rows(one, 1, l9);
  EXPECT(b.state == READY && b.len[1] == 9 && b.len[2] == 50);
  // append: len + n <= capacity exactly (no scratch positions needed)
  int32_t fit[4] = {118, 0, 78, 98};
  EXPECT(b.check_append(fit, e) == S_OK);
  int32_t over[4] = {119, 0, 0, 0};
  EXPECT(b.check_append(over, e) == S_ECAPACITY);
  int32_t neg[4] = {0, -1, 0, 0};
  EXPECT(b.check_append(neg, e) == S_EINVAL);
  EXPECT(b.check_append(nullptr, e) == S_EINVAL);
  b.commit_new(fit);
  EXPECT(b.len[0] == 128 && b.len[1] == 9 && b.len[2] == 128 && b.len[3] == 128);
  // a whole-context invalidate marks every row; a full build restores all
  b.invalidate();
  EXPECT(b.state == INVALID && b.row_state[1] == INVALID);
  int32_t all[4] = {5, 6, 7, 8};
  b.commit_build(all);
  EXPECT(b.state == READY && b.row_state[3] == READY && b.len[3] == 8);
}

// Shared prefix pages: reference counts, the key index, attach / publish / free.
static void test_pages() {
  PagePool pool;
  pool.init(12);
  EXPECT(pool.in_use() == 0 && pool.alloc() == 0 && pool.alloc() == 1 && pool.in_use() == 2);
  pool.publish(1, 77);
  EXPECT(pool.lookup(77) == 1 && pool.lookup(78) == -1);
  pool.retain(1);
  pool.release(1);
  EXPECT(pool.refs[1] == 1 && pool.lookup(77) == 1);  // still referenced: stays indexed
  pool.release(1);
  EXPECT(pool.refs[1] == 0 && pool.lookup(77) == -1 && pool.in_use() == 1);  // freed at zero
  pool.release(0);
  EXPECT(pool.in_use() == 0);

  // 3 rows of 3 pages; rows 0 and 1 agree on their first two pages, row 2 on the first
  const int ppr = 3;
  pool.init(9);
  std::vector<int32_t> pt(3 * ppr, -1), start;
  std::string e;
  int32_t rows[3] = {0, 1, 2}, share[3] = {2, 2, 2};
  uint64_t keys[9] = {10, 11, 0, 10, 11, 0, 10, 12, 0};
  EXPECT(plan_row_pages(pool, pt, ppr, rows, 3, share, keys, ppr, true, start, e) == S_OK);
  EXPECT(pt[0] == pt[3] && pt[1] == pt[4] && pt[2] != pt[5]);  // row 1 attaches row 0's two pages
  EXPECT(pt[6] == pt[0] && pt[7] != pt[1]);                    // row 2 attaches only the first
  EXPECT(start[0] == 0 && start[1] == 128 && start[2] == 64);
  EXPECT(pool.refs[pt[0]] == 3 && pool.refs[pt[1]] == 2 && pool.refs[pt[7]] == 1);
  EXPECT(pool.in_use() == 3 + 1 + 2);  // row 0: 3 pages; row 1: its last; row 2: its last two
  EXPECT(pool.lookup(12) == pt[7]);                // row 2 published the page it computed
  // without sharing every row takes fresh pages: the pool of 9 is then full
  PagePool p2;
  p2.init(9);
  std::vector<int32_t> pt2(3 * ppr, -1);
  EXPECT(plan_row_pages(p2, pt2, ppr, rows, 3, share, keys, ppr, false, start, e) == S_OK);
  EXPECT(p2.in_use() == 9 && start[1] == 0 && p2.lookup(10) == -1);
  // a pool too small: ECAPACITY, nothing changed
  PagePool p3;
  p3.init(5);
  std::vector<int32_t> pt3(3 * ppr, -1);
  EXPECT(plan_row_pages(p3, pt3, ppr, rows, 3, share, keys, ppr, true, start, e) == S_ECAPACITY);
  EXPECT(p3.in_use() == 0 && pt3[0] == -1 && !e.empty());
  // row 0 invalidated: its pages lose a reference; the shared ones stay with rows 1 and 2
  int32_t r0[1] = {0};
  const int first = pt[0], own0 = pt[2];
  release_row_pages(pool, pt, ppr, r0, 1);
  EXPECT(pool.refs[first] == 2 && pool.refs[own0] == 0 && pt[0] == -1 && pool.lookup(10) == first);
  // rebuilt with a different first page: nothing to attach, three fresh pages
  uint64_t k0[3] = {20, 21, 0};
  int32_t s0[1] = {2};
  EXPECT(plan_row_pages(pool, pt, ppr, r0, 1, s0, k0, ppr, true, start, e) == S_OK);
  EXPECT(start[0] == 0 && pt[0] != first && pool.lookup(20) == pt[0]);
  // every row released: the pool is empty and the index too
  release_row_pages(pool, pt, ppr, rows, 3);
  EXPECT(pool.in_use() == 0 && pool.index.empty());
  EXPECT(shareable_pages(64) == 0 && shareable_pages(65) == 1 && shareable_pages(128) == 1 && shareable_pages(300) == 4);
  EXPECT(page_key_segment(8192) == 4096 && page_key_segment(768) == 256 && page_key_segment(512) == 512);
}

// Rows moved to host memory: OFFLOADED until reloaded; only READY rows offload,
// only rows not READY reload.
static void test_offload_states() {
  RowBook b;
  b.init(3, 128);
  std::string e;
  int32_t lens[3] = {10, 20, 30};
  b.commit_build(lens);
  int32_t r1[1] = {1};
  EXPECT(b.check_reload(r1, 1, e) == S_ESTATE);  // READY rows are not reloaded
  EXPECT(b.check_offload(r1, 1, e) == S_OK);
  b.offload_rows(r1, 1);
  EXPECT(b.row_state[1] == OFFLOADED && b.len[1] == 0 && b.state == INVALID);
  EXPECT(b.check_offload(r1, 1, e) == S_ESTATE);  // nothing left to offload
  EXPECT(b.check_step(nullptr, 1, e) == S_ESTATE);
  EXPECT(b.check_reload(r1, 1, e) == S_OK);
  int32_t l1[1] = {20};
  b.commit_build_rows(r1, 1, l1);
  EXPECT(b.state == READY && b.len[1] == 20);
  // tier plan: priority first, LRU within it, pinned and non-resident rows kept
  int32_t prio[5] = {1, 0, 0, 2, 0}, pages[5] = {4, 2, 3, 8, 1}, drop[5] = {0, 1, 0, 0, 1};
  int32_t res[5] = {1, 1, 1, 1, 0}, pin[5] = {0, 0, 0, 0, 0}, act[5];
  int64_t last[5] = {5, 9, 3, 1, 3};
  EXPECT(tier_plan(5, prio, last, pages, drop, res, pin, 4, act) == 5);
  EXPECT(act[0] == TIER_KEEP && act[1] == TIER_DROP && act[2] == TIER_OFFLOAD && act[3] == TIER_KEEP &&
         act[4] == TIER_KEEP);
  EXPECT(tier_plan(5, prio, last, pages, drop, res, pin, 0, act) == 0 && act[2] == TIER_KEEP);
}

static void test_plan() {
  // rows 0..5 with ragged counts, one empty; pass budget 100
  int32_t counts[6] = {40, 0, 70, 30, 100, 1};
  int32_t start[6] = {0, 0, 5, 7, 0, 9};
  Plan p = plan_passes(6, counts, start, 100);
  // passes: [r0] (40, next 70 overflows) [r2, r3] (100) [r4] (100) [r5] (1)
  EXPECT(p.passes.size() == 4);
  EXPECT(p.row.size() == 5);
  int tok = 0, seg = 0;
  for (size_t i = 0; i < p.passes.size(); ++i) {
    const Pass& ps = p.passes[i];
    EXPECT(ps.seg_begin == seg);
    EXPECT(ps.tok_src == tok);
    const int32_t* off = p.off.data() + ps.seg_begin + i;
    EXPECT(off[0] == 0);
    int sum = 0, mx = 0, me = 0;
    for (int s = 0; s < ps.n_seg; ++s) {
      const int r = p.row[ps.seg_begin + s];
      EXPECT(off[s + 1] - off[s] == counts[r]);
      EXPECT(p.pos[ps.seg_begin + s] == start[r]);
      sum += counts[r];
      mx = std::max(mx, counts[r]);
      me = std::max(me, start[r] + counts[r]);
    }
    EXPECT(sum == ps.n_tok && ps.n_tok <= 100);
    EXPECT(mx == ps.max_len && me == ps.max_end);
    tok += ps.n_tok;
    seg += ps.n_seg;
  }
  EXPECT(tok == 241);
  EXPECT(p.off.size() == p.row.size() + p.passes.size());
  int32_t none[3] = {0, 0, 0};
  EXPECT(plan_passes(3, none, none, 64).passes.empty());
}

static void test_layout() {
  Cfg c{12, 1024, 16, 64, 4096, 256, 256, 1e-5f, 10000.f, 1};
  std::string e;
  EXPECT(check_cfg(c, e) == S_OK);
  const ModelLayout m = model_layout(c);
  EXPECT(m.per_layer_qkv == 3ull * 1024 * 1024 * 2);
  EXPECT(m.total >= 12ull * (4 * 1024 * 1024 + 3 * 1024 * 4096) * 2);
  const CtxLayout x = ctx_layout(c, 8, 320, 0);
  EXPECT(x.slab_layer == 8ull * 320 * 1024 * 2);
  EXPECT(x.kv == 0 && x.h >= 2ull * 12 * x.slab_layer);
  EXPECT(x.pass_tokens == 2560 && x.total % 256 == 0);
  size_t offs[] = {x.kv, x.h, x.u, x.qkv, x.o, x.a, x.h_last, x.part, x.logits, x.rope, x.lens, x.meta, x.total};
  for (size_t i = 0; i + 1 < sizeof(offs) / sizeof(offs[0]); ++i) EXPECT(offs[i] < offs[i + 1] && offs[i] % 256 == 0);
  Cfg bad = c;
  bad.head_dim = 96; bad.n_heads = 1024 / 96;
  EXPECT(check_cfg(bad, e) == S_EINVAL);
  bad = c; bad.d_ffn = 4000;
  EXPECT(check_cfg(bad, e) == S_EINVAL);
  bad = c; bad.n_bins = 300;
  EXPECT(check_cfg(bad, e) == S_EINVAL);
  bad = c; bad.rms_eps = 0.f;
  EXPECT(check_cfg(bad, e) == S_EINVAL);
  EXPECT(check_ctx_args(c, 0, 320, 0, e) == S_EINVAL);
  EXPECT(check_ctx_args(c, 8, 100, 0, e) == S_EINVAL);
  EXPECT(check_ctx_args(c, 8, 320, 100, e) == S_EINVAL);
  EXPECT(check_ctx_args(c, 8, 320, 320, e) == S_OK);
  EXPECT(decode_splits(1, 32, 320) == 1);    // short context: one workgroup per pair
  EXPECT(decode_splits(1, 32, 2048) == 1);
  EXPECT(decode_splits(1, 32, 4096) == 4);   // long context, 32 pairs: parts of >= 1024
  EXPECT(decode_splits(1, 32, 16384) == 8);  // 32 pairs x 8 = 256 workgroups
  EXPECT(decode_splits(8, 16, 8192) == 1);   // 128 pairs: no split
  EXPECT(decode_splits(64, 32, 768) == 1);
  EXPECT(decode_splits(1, 1, 64) == 1);
  EXPECT(bins_padded(c) == 256);
}

int main() {
  test_book();
  test_async_error();
  test_rows();
  test_pages();
  test_offload_states();
  test_plan();
  test_layout();
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("state_test: ok\n");
  return 0;
}

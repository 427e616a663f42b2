// Host unit test of the KV pool bookkeeping (block_pool.h), built with the
// address and undefined-behaviour sanitizers by tests/test_block_pool_host.py.
// Random sequences of prefills (ensure from 0), commits (ensure to a longer
// length, copy-at-commit index mapping) and releases over several handles
// are checked against the invariants: every block is either free or owned
// by exactly one handle, tables point only at owned blocks, exhaustion and
// the context limit are reported, and a commit's copy lands on the blocks
// the prefix owns at the right slots.
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <random>
#include <set>
#include <vector>

#include "block_pool.h"

using cdsl::BlockPool;
using cdsl::kPoolBlock;

#define CHECK(x)                                                        \
  do {                                                                  \
    if (!(x)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x);   \
      exit(1);                                                          \
    }                                                                   \
  } while (0)

struct Handle {
  int B = 0;
  std::vector<int> table, owned, len;
  bool live = false;
};

static void check_invariants(const BlockPool& pool, const std::vector<Handle>& hs, int first, int last, int pstride) {
  std::set<int> owned;
  size_t n_owned = 0;
  for (const Handle& h : hs) {
    if (!h.live) continue;
    for (int blk : h.owned) {
      CHECK(blk >= first && blk < last);
      CHECK(owned.insert(blk).second);     // owned by one handle, once
    }
    n_owned += h.owned.size();
    std::set<int> mine(h.owned.begin(), h.owned.end());
    for (int b = 0; b < h.B; ++b) {
      const int need = (h.len[b] + kPoolBlock - 1) / kPoolBlock;
      for (int q = 0; q < pstride; ++q) {
        const int blk = h.table[(size_t)b * pstride + q];
        if (q < need) CHECK(blk >= 0);
        if (blk >= 0) CHECK(mine.count(blk) == 1);
      }
    }
  }
  CHECK((int)n_owned + pool.available() == last - first);
}

int main() {
  std::mt19937 rng(12345);
  const int suffix_blocks = 24, pstride = 9;
  for (int round = 0; round < 200; ++round) {
    const int last = suffix_blocks + 20 + (int)(rng() % 60);
    BlockPool pool;
    pool.reset(suffix_blocks, last);
    std::vector<Handle> hs(4);
    for (int op = 0; op < 300; ++op) {
      Handle& h = hs[rng() % hs.size()];
      if (!h.live) {                       // prefill
        h.B = 1 + (int)(rng() % 3);
        h.table.assign((size_t)h.B * pstride, -1);
        h.owned.clear();
        h.len.assign(h.B, 0);
        h.live = true;
        for (int b = 0; b < h.B; ++b) {
          const int L = 1 + (int)(rng() % 40);
          const int r = pool.ensure(h.table, h.owned, pstride, b, L);
          if (r == BlockPool::kOk) h.len[b] = L;
          else CHECK(r == BlockPool::kExhausted);
        }
      } else if (rng() % 5 == 0) {         // free the handle
        pool.release(h.owned);
        CHECK(h.owned.empty());
        h.live = false;
      } else {                             // commit of ne tokens to prompt b
        const int b = (int)(rng() % h.B);
        const int ne = (int)(rng() % 12);
        const int soff = (int)(rng() % 2);
        const int newlen = h.len[b] + ne;
        const int r = pool.ensure(h.table, h.owned, pstride, b, newlen);
        if (newlen > pstride * kPoolBlock) {
          CHECK(r == BlockPool::kRange);
        } else if (r == BlockPool::kOk) {
          // the copy of slots soff .. soff + ne - 1 of a beam with two
          // suffix blocks lands on owned prefix blocks at the new positions
          const int srow[2] = {(int)(rng() % suffix_blocks), (int)(rng() % suffix_blocks)};
          std::set<int> mine(h.owned.begin(), h.owned.end());
          for (int t = 0; t < ne && t + soff < 2 * kPoolBlock; ++t) {
            const cdsl::PromoteIndex ix = cdsl::promote_index(srow, &h.table[(size_t)b * pstride], h.len[b], t, soff);
            CHECK(ix.sblk == srow[(t + soff) / kPoolBlock] && ix.sslot == (t + soff) % kPoolBlock);
            CHECK(mine.count(ix.pblk) == 1);
            CHECK(ix.pblk == h.table[(size_t)b * pstride + (h.len[b] + t) / kPoolBlock]);
            CHECK(ix.pslot == (h.len[b] + t) % kPoolBlock);
          }
          h.len[b] = newlen;
        } else {
          CHECK(r == BlockPool::kExhausted);
        }
      }
      check_invariants(pool, hs, suffix_blocks, last, pstride);
    }
    for (Handle& h : hs)
      if (h.live) pool.release(h.owned);
    CHECK(pool.available() == last - suffix_blocks);
  }
  // an exhausted pool, then the same request after a release
  BlockPool pool;
  pool.reset(0, 2);
  std::vector<int> t1(4, -1), o1, t2(4, -1), o2;
  CHECK(pool.ensure(t1, o1, 4, 0, 2 * kPoolBlock) == BlockPool::kOk);
  CHECK(pool.ensure(t2, o2, 4, 0, 1) == BlockPool::kExhausted);
  pool.release(o1);
  CHECK(pool.ensure(t2, o2, 4, 0, 1) == BlockPool::kOk && o2.size() == 1);
  CHECK(pool.ensure(t2, o2, 4, 0, 4 * kPoolBlock + 1) == BlockPool::kRange);
  printf("block pool: ok\n");
  return 0;
}

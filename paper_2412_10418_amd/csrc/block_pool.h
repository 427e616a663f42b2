// Bookkeeping of the paged KV pool, host side, plus the index mapping of a
// commit's copy from a beam's suffix slots into the prefix (shared with the
// promote kernels).  Plain C++ without HIP headers, so that it also builds
// as host-only code for unit tests under the address and undefined-behaviour
// sanitizers.
//
// Blocks hold kPoolBlock consecutive token positions of one prompt (all
// layers and KV heads; the device arrays are indexed by the block id).
// Ids [0, suffix_blocks) are the fixed per-(prompt, beam) suffix blocks of
// the lookahead rows; ids [suffix_blocks, nblocks) are handed out to the
// prefixes from a free list.  A prefix handle keeps, per prompt, a table of
// pstride block ids (position p lives in table[p / kPoolBlock], -1 = not
// yet owned) and the list of blocks it owns, returned on release.
#pragma once

#include <stdint.h>

#include <vector>

#if defined(__HIPCC__)
#define CDSL_HD __host__ __device__
#else
#define CDSL_HD
#endif

namespace cdsl {

constexpr int kPoolBlock = 16;

class BlockPool {
 public:
  enum { kOk = 0, kRange = 1, kExhausted = 2 };

  // ids [first, last) become free; lower ids are handed out first
  void reset(int first, int last) {
    free_.clear();
    free_.reserve(last > first ? last - first : 0);
    for (int u = last - 1; u >= first; --u) free_.push_back(u);
  }

  int available() const { return (int)free_.size(); }

  // Make prompt b of a table [B][pstride] own blocks for positions
  // [0, new_len).  New blocks go to `owned`.  kRange when new_len needs
  // more than pstride blocks, kExhausted when the free list runs out (the
  // blocks taken before that stay owned and valid).
  int ensure(std::vector<int>& table, std::vector<int>& owned, int pstride, int b, int new_len) {
    const int need = (new_len + kPoolBlock - 1) / kPoolBlock;
    if (need > pstride) return kRange;
    for (int q = 0; q < need; ++q) {
      int& slot = table[(size_t)b * pstride + q];
      if (slot >= 0) continue;
      if (free_.empty()) return kExhausted;
      slot = free_.back();
      free_.pop_back();
      owned.push_back(slot);
    }
    return kOk;
  }

  // Give back every block of a handle.
  void release(std::vector<int>& owned) {
    for (int blk : owned) free_.push_back(blk);
    owned.clear();
  }

 private:
  std::vector<int> free_;
};

// Source and destination of token t of a commit's copy into the prefix:
// suffix slot t + soff of beam i (its blocks: srow[0 ..]) goes to prefix
// position L0 + t (the prompt's table row prow).
struct PromoteIndex {
  int sblk, sslot, pblk, pslot;
};

CDSL_HD inline PromoteIndex promote_index(const int* srow, const int* prow, int L0, int t, int soff) {
  PromoteIndex r;
  r.sblk = srow[(t + soff) / kPoolBlock];
  r.sslot = (t + soff) % kPoolBlock;
  const int pos = L0 + t;
  r.pblk = prow[pos / kPoolBlock];
  r.pslot = pos % kPoolBlock;
  return r;
}

}  // namespace cdsl

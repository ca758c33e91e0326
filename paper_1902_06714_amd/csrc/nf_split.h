// Host-side arithmetic of the k-range pieces of a contraction (plain C++, no
// HIP): how a forward contraction's input range is cut, and the alignment
// every piece must keep when an operand is loaded 16 bytes at a time along k.
//
// Piece z = shard * nsub + sub of a contraction covers the k range
//   [shard * shard_len + sub * sub_len, min(that + sub_len, (shard + 1) * shard_len)).
// A k-contiguous operand read with 16-byte vectors loads VW = 16 / sizeof(T)
// consecutive k at a time, from k0 + 4j within a stage of BK = 16 starting at
// the piece's first k.  Were a piece to start off a multiple of VW, its loads
// would be misaligned, and the last vector of the piece before it would run
// past that piece's end into the next piece's first elements (counted twice)
// and, in the last row of the operand, past the end of the row.  So every
// piece of such an operand starts on a whole stage of BK elements.
#pragma once

#include <stdint.h>

namespace nf {

constexpr int KSPLIT_BK = 16;   // k per operand stage of the contraction

struct KSplit {
  int nsplit;    // pieces actually used
  int sub_len;   // k per piece (the last may be shorter), a multiple of KSPLIT_BK
};

// The cut of [0, K) into at most `want` pieces on whole stages.
inline KSplit k_split(int64_t K, int64_t want) {
  KSplit r{1, (int)K};
  if (K <= 0 || want <= 1) return r;
  const int64_t per = (K + want - 1) / want;
  const int64_t sub = (per + KSPLIT_BK - 1) / KSPLIT_BK * KSPLIT_BK;
  r.sub_len = (int)sub;
  r.nsplit = (int)((K + sub - 1) / sub);
  return r;
}

// Every piece boundary inside [0, K) lies on a whole stage: true when the
// shard length (if there is more than one shard) and the piece length (if a
// shard holds more than one piece) are multiples of KSPLIT_BK.
inline bool k_pieces_aligned(int nshards, int64_t shard_len, int nsub, int64_t sub_len) {
  if (nshards > 1 && shard_len % KSPLIT_BK != 0) return false;
  if (nsub > 1 && sub_len % KSPLIT_BK != 0) return false;
  return true;
}

}  // namespace nf

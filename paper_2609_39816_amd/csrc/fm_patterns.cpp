// Run-time matching of a scheme's coefficient lists against the nonzero
// structures that have specialized kernels (fm_patterns.inc).
#include <cstring>

#include "fm_internal.h"
#include "fm_patterns.inc"

namespace fm {
namespace {

struct PatternRef {
  const char* name;
  int R;
  int nb[3];
  int nnz[3];
  const int16_t* rowptr[3];
  const int16_t* idx[3];
  bool joint;  // H pattern generated (at most 64 products)
  int hnnz;
  const int16_t* hrowptr;
  const int16_t* hidx;
  bool trie[2];             // prefix-shared chains generated (A, B)
  const uint32_t* val[2];   // the base scheme's coefficient bits per list entry
};

#define FM_PATTERN_REF(P)                                                    \
  PatternRef{#P,                                                             \
             pat::P::R,                                                      \
             {pat::P::A::NB, pat::P::B::NB, pat::P::W::NB},                  \
             {pat::P::A::NNZ, pat::P::B::NNZ, pat::P::W::NNZ},               \
             {pat::P::A::rowptr, pat::P::B::rowptr, pat::P::W::rowptr},      \
             {pat::P::A::idx, pat::P::B::idx, pat::P::W::idx},                \
             pat::P::H::JOINT,                                               \
             pat::P::H::NNZ,                                                 \
             pat::P::H::rowptr,                                              \
             pat::P::H::idx,                                                 \
             {pat::P::A::TRIE, pat::P::B::TRIE},                             \
             {pat::P::A::val, pat::P::B::val}},

const PatternRef kPatterns[] = {FM_PATTERN_FAMILIES(FM_PATTERN_REF)};
constexpr int kNumPatterns = sizeof(kPatterns) / sizeof(kPatterns[0]);

}  // namespace

int pattern_count() { return kNumPatterns; }

const char* pattern_name(int id) {
  return (id >= 0 && id < kNumPatterns) ? kPatterns[id].name : "generic";
}

int match_pattern(int side, const Side& s, int R, int NB) {
  for (int p = 0; p < kNumPatterns; ++p) {
    const PatternRef& P = kPatterns[p];
    if (P.R != R || P.nb[side] != NB || P.nnz[side] != (int)s.idx.size()) continue;
    bool ok = true;
    for (int r = 0; r <= R && ok; ++r) ok = (P.rowptr[side][r] == s.off[r] - s.off[0]);
    for (size_t e = 0; e < s.idx.size() && ok; ++e) ok = (P.idx[side][e] == s.idx[e]);
    if (ok) return p;
  }
  return -1;
}

bool block_signs(int pattern, int side, const Side& s, int NB, uint64_t* mask) {
  if (pattern < 0 || pattern >= kNumPatterns || side < 0 || side > 1 || NB > 64) return false;
  const PatternRef& P = kPatterns[pattern];
  if (!P.trie[side] || (int)s.coef.size() != P.nnz[side]) return false;
  // every coefficient must be its base value with the sign of its block:
  // equal bits, or bits differing in the sign alone, the same way for
  // every entry of a block (entries index one scheme's list, s.off[0] == 0)
  uint64_t neg = 0, seen = 0;
  for (size_t e = 0; e < s.coef.size(); ++e) {
    const int b = s.idx[e];
    if (b < 0 || b >= NB) return false;
    uint32_t c;
    std::memcpy(&c, &s.coef[e], 4);
    const uint32_t diff = c ^ P.val[side][e];
    if (diff != 0u && diff != 0x80000000u) return false;
    const uint64_t bit = (uint64_t)1 << b;
    const uint64_t flip = diff ? bit : 0;
    if ((seen & bit) && (neg & bit) != flip) return false;
    seen |= bit;
    neg |= flip;
  }
  *mask = neg;
  return true;
}

int match_h_pattern(const int32_t* rowptr, const uint16_t* cols, int R) {
  for (int p = 0; p < kNumPatterns; ++p) {
    const PatternRef& P = kPatterns[p];
    if (!P.joint || P.R != R || P.hnnz != rowptr[R]) continue;
    bool ok = true;
    for (int r = 0; r <= R && ok; ++r) ok = P.hrowptr[r] == rowptr[r];
    for (int e = 0; e < P.hnnz && ok; ++e) ok = P.hidx[e] == (int)cols[e];
    if (ok) return p;
  }
  return -1;
}

}  // namespace fm

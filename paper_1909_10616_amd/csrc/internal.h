// Internal declarations shared by the library's translation units.
#pragma once
#include <cstdint>
#include <string>

#include "gemmtune.h"

namespace gt {

void set_error(const std::string& msg);

// One dimension of the space: extent D = q·2^E, d levels (§3.3 Eq.2–4).
struct Dim {
  int64_t D = 1, q = 1;
  int E = 0, d = 1;
  uint64_t count = 1;  // C(E + d − 1, d − 1)
};

struct Space {
  Dim dim[3];  // m, k, n
  uint64_t n_mfma = 1;
  uint64_t size = 1;
  int dtype = GT_F32;   // gt_dtype without the layout flag
  bool a_kmajor = false;  // GT_A_KMAJOR: A given as its K×M transpose
  int mfma_coord = 0;
  int mode = GT_ADJACENT;
  int64_t ext[3] = {1, 1, 1};
};

// Validates and fills a Space; GT_OK or GT_EINVAL (message set).
int make_space(const gt_space* sp, Space* s);
bool is_member(const Space& s, const gt_config& c);
uint64_t rank_of(const Space& s, const gt_config& c);  // requires is_member
void unrank_into(const Space& s, uint64_t rank, gt_config* c);
int legit_of(const Space& s, const gt_config& c);
// Ranks [start, start + n) (within the space) into out[0 .. n), J filled.
void enumerate_range(const Space& s, uint64_t start, uint64_t n, gt_config* out);
// g(s) in ascending rank with J filled; returns the count (≤ kMaxNeighbours).
constexpr int kMaxNeighbours = 3 * GT_MAXD * (GT_MAXD - 1) + 1;
int neighbour_list(const Space& s, const gt_config& c, gt_config* out);

// The hardware meaning of a configuration's levels (level 0 outermost).
struct Levels {
  int64_t gridM, wavesM, repM, blkM;
  int64_t gridN, wavesN, repN, blkN;
  int64_t kLoop, kSplit, kSub, kBlk;
  int I, IK;        // MFMA size and K per instruction
  int64_t TM, TN;   // MFMA tiles per wavefront
  int64_t acc;      // accumulator registers per lane
  int64_t W;        // wavefronts per workgroup
  int64_t BM, BN, BK;
  int elem;         // bytes per input element
};
void levels_of(const gt_config& c, int dtype, Levels* L);

constexpr int64_t kLdsMax = 163840;  // gfx950 LDS per workgroup

}  // namespace gt

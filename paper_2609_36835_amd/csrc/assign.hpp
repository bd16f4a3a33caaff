// Work lists of the certified key-to-anchor assignment (assign.hip), shared by
// the kernels and the host-side stage sequencing.  All pointers are device
// arrays for one chunk of P pairs.
#pragma once
#include <stdint.h>

namespace arckv {

constexpr int kAssignStats = 8;

struct AssignLists {
  int32_t *fcnt;    // [P] keys queued for the refine pass
  int32_t *fkey;    // [P][cap]
  int32_t *foff;    // [P][cap] first candidate of the queued key in the pool
  int32_t *fn;      // [P][cap] its number of candidates
  int32_t *pcnt;    // [P] candidates in the pool
  int32_t *pool;    // [P][pcap] candidate anchors, contiguous per queued key
  double *psim;     // [P][pcap] their refined similarities
  int64_t pcap;     // pool capacity per pair
  int32_t *dcnt;    // [P] keys queued for the float64 pass
  int32_t *dkey;    // [P][cap]
  int32_t *dn;      // [P][cap] entries per queued key
  int32_t *doff;    // [P][cap] first surviving candidate of the queued key in the pool (-1: all t anchors)
  int32_t *stats;   // [P][kAssignStats] (assign.hip): flagged after the first pass, sent to the float64
                    // pass, candidates of the flagged keys, undecided (sum of the next two), undecided
                    // in the first pass, undecided in the refine pass (kept at 0: survivors of any
                    // number go to the float64 pass), sent to the refine pass, keys whose pass-A
                    // candidates include a whole anchor tile
  int64_t cap;      // key capacity per pair
  int32_t *goff;    // [P][gcap] pass C work items: first (group of 64 queued keys, candidate chunk) item of each
                    // group, then the pair's item count
  int64_t gcap;     // >= cap / 64 + 1
};

}  // namespace arckv

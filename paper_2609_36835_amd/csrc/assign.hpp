// Work lists of the certified key-to-anchor assignment (assign.hip), shared by
// the kernels and the host-side stage sequencing.  All pointers are device
// arrays for one chunk of P pairs.
#pragma once
#include <stdint.h>

namespace arckv {

constexpr int kAssignStats = 8;

// Pool survivors per float64-pass entry: a key and 31 candidates fill one
// batch of 32 vectors.  A key with more pool survivors is queued as several
// entries, so its batches can run on different workgroups.
constexpr int kPassDSplit = 31;

// Entries for at most Tp queued keys whose pool candidates number at most
// pool_per_key * Tp: one per key, plus one per kPassDSplit candidates of a
// split key.
inline int64_t pass_d_capacity(int64_t Tp, int64_t pool_per_key) {
  return Tp + (pool_per_key * Tp + kPassDSplit - 1) / kPassDSplit + 1;
}

struct AssignLists {
  int32_t *fcnt;    // [P] keys queued for the refine pass
  int32_t *fkey;    // [P][cap]
  int32_t *foff;    // [P][cap] first candidate of the queued key in the pool
  int32_t *fn;      // [P][cap] its number of candidates
  int32_t *pcnt;    // [P] candidates in the pool
  int32_t *pool;    // [P][pcap] candidate anchors, contiguous per queued key
  double *psim;     // [P][pcap] their refined similarities
  int64_t pcap;     // pool capacity per pair
  int32_t *dcnt;    // [P] entries queued for the float64 pass (a key with many pool survivors is split
                    // into several entries of consecutive survivors)
  int32_t *dkey;    // [P][dcap] the entry's key
  int32_t *dn;      // [P][dcap] candidates of the entry
  int32_t *doff;    // [P][dcap] its first candidate in the pool (-1: all t anchors)
  int32_t *stats;   // [P][kAssignStats] (assign.hip): flagged after the first pass, sent to the float64
                    // pass, candidates of the flagged keys, undecided (sum of the next two), undecided
                    // in the first pass, undecided in the refine pass (kept at 0: survivors of any
                    // number go to the float64 pass), sent to the refine pass, keys whose pass-A
                    // candidates include a whole anchor tile
  int64_t cap;      // key capacity per pair
  int32_t *goff;    // [P][gcap] pass C work items: first (group of 64 queued keys, candidate chunk) item of each
                    // group, then the pair's item count
  int64_t gcap;     // >= cap / 64 + 1
  int32_t *dgrp;    // [P][dcap] first entry of the entry's key when the key is split, else -1
  int32_t *dgn;     // [P][dcap] entries of the entry's key
  double *dsim;     // [P][dcap] best similarity of a split entry's candidates
  int32_t *dr;      // [P][dcap] its anchor
  int32_t *ditem;   // [P][dcap + 2] pass D work items: count, first entry of each item, then dcnt
  int64_t dcap;     // entry capacity per pair
};

}  // namespace arckv

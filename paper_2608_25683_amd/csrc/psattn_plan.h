// Work-plan records shared by the host planner and the HIP kernels.
//
// A plan turns a prefix forest into three lists of independent work items:
//   * forward / dQ items: a tile of query rows of one node (or a piece of
//     its key range) x the node's root-to-node key path x a chunk of query
//     heads that read one kv head;
//   * dK/dV items: a tile of keys of one node x one kv head x a chunk of the
//     rows that consume those keys: every row of every descendant node (all
//     branches reusing the prefix), then the node's own rows from its last
//     position down to the tile's first key.  All tiles of a node therefore
//     read the same rows in the same order, and their concurrent workgroups
//     share those rows in L2;
//   * fixed-order merge/reduce lists for items whose results are split.
// Keys are addressed through per-path lists of pool slots, so a key tile
// can straddle page blocks of any size.
#pragma once
#include <stdint.h>

namespace psattn {

constexpr int KV_TILE = 64;    // keys per forward / dQ key tile
constexpr int Q_SUB = 32;      // query rows per wavefront subtile
constexpr int BKV_TILE = 128;  // keys per dK/dV work item (4 wavefronts x 32 keys)

struct FwdItem {     // also the dQ item
  int32_t q_off;     // first entry in q_list (packed row indices)
  int32_t nq;        // rows in the tile, 1..q_tile_rows
  int32_t kv_off;    // entry in kv_list holding the slot of the first key
  int32_t nkv;       // keys in this item's range, >= 1
  int32_t kv_pos0;   // sequence position of the first key
  int32_t head0;     // first query head of the chunk
  int32_t part;      // -1: write final results; else first partial row
  int32_t nfull;     // leading key tiles that need no mask
};

struct MergeEntry {  // a query tile whose key range was split into pieces
  int32_t q_off, nq;
  int32_t part0;     // piece j writes partial rows part0 + j*q_tile_rows + i
  int32_t nparts;
};

struct BkvItem {
  int32_t kv_off;    // entry in kv_list holding the slot of the first key
  int32_t nk;        // keys, 1..BKV_TILE
  int32_t kv_pos0;   // sequence position of the first key
  int32_t q_off;     // first consumer row (entry in q_list)
  int32_t nq;        // consumer rows in this chunk
  int32_t hk;        // kv head
  int32_t part;      // -1: write dK/dV directly; else partial tile index
  int32_t mask_lo;   // chunk rows [mask_lo, mask_hi) may see only part of the keys;
  int32_t mask_hi;   //   every other row sees all of them
  int32_t acc;       // 1: a cached (external) node's keys: add to dK/dV instead of writing them
};

struct ReduceEntry {  // a key tile whose consumer rows were split into chunks
  int32_t kv_off, nk, hk;
  int32_t part0;      // chunk j wrote partial tile part0 + j
  int32_t nparts;
  int32_t acc;        // 1: add the sum to dK/dV (a cached node's keys)
  int32_t pad[2];
};

// Device-side view of an uploaded plan.
struct PlanView {
  const int32_t* row_pos;   // [Ns] sequence position of each packed row
  const int32_t* row_slot;  // [Ns] pool slot of each packed row's K/V
  const int32_t* q_list;
  const int32_t* q_pos;     // sequence position of each q_list entry; q_pos[-1] = -1
  const int32_t* kv_list;
  const FwdItem* fwd;
  const MergeEntry* merge;
  const BkvItem* bkv;
  const ReduceEntry* reduce;
  const int32_t* pad_slots;
};

// Problem shape handed to every launcher.
struct Shape {
  int32_t ns;       // packed rows
  int32_t hq, hkv, d;
  int32_t g;        // hq / hkv
  int32_t hc;       // query heads per forward item
  int32_t rw;       // 32-row subtiles per head in a forward item
  int32_t nw;       // wavefronts per forward workgroup = hc * rw
  int32_t bmq;      // query rows per forward item = 32 * rw
  float scale;
};

}  // namespace psattn

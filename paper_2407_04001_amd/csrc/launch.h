// Host-side description of one search's launches (no HIP): the per-vertex
// kernel descriptors, the batched launches of each launch slot, and the
// constant-region image uploaded before the first kernel.  Built by
// launch_plan.cpp against a workspace base address; the device runtime only
// uploads the image and enqueues the batches.
#pragma once

#include <cstdint>
#include <vector>

#include "internal.h"

namespace pase {

// One vertex's kernel descriptors, resolved against the workspace base.
template <typename KeyT>
struct Launch {
    PrepArgs prep;
    bool rows = false;
    bool direct = false;
    bool fused = false;    // a fused minimum: its fill is the one-split reduction `red`
    RowsArgs ra;
    GenericArgs ga;
    ReduceArgs red;
    DirectArgs da;
};

// A batched launch: vertices (sequence positions) sharing one kernel variant
// within one launch group, with their first workgroups.
struct Batch {
    enum Kind { kPrep, kRows, kGeneric, kReduce, kDirect } kind;
    int lane;              // bulk lane schedule: the stream it runs on (0 = the caller's)
    int group;             // launch group (a slot, or a (slot, lane) pair) it belongs to
    uint32_t variant;      // rows: (TZ * 4 + TM) * 8 + NA (NA 7 = runtime count); generic: NT (0 = runtime)
    uint32_t entry0;       // first BatchEntry of this batch
    uint32_t nentries;
    uint32_t blocks;       // workgroups of the launch
    bool side = false;     // a hoisted prep launch: on the side stream, after the work enqueued before it
};

constexpr int kLanes = 2;   // streams of the bulk lane and split chains schedules

struct SearchImage {
    std::vector<Batch> batches;            // in enqueue order
    std::vector<std::vector<int>> groups;  // positions of each launch group
    std::vector<int> group_lane;           // lane of each launch group
    bool lanes = false;                    // a lane schedule runs (one stream per lane in use)
    bool hoist = false;                    // hoisted preps run on a side stream (level layout)
    bool lane_hoist = false;               // hoisted preps run early on their vertex's lane (lanes)
    std::vector<std::vector<int>> group_waits;   // per launch group: the side batches it waits for
    bool upload_costs = true;              // the device cost tables' range is part of the upload
    uint32_t nlev = 0;                     // backward levels of the back-substitution
    uint64_t nL = 0;                       // layer costs of all vertices (sum of K)
};

// Kernel descriptors of every position; contributions in upload order.
template <typename KeyT>
pase_status build_launches(pase_graph_t g, char *ws, std::vector<Launch<KeyT>> &out,
                           std::vector<Contrib> &contrib);

// The constant-region image [0, plan.off_cfg) of one search into `img` (host
// memory of at least plan.off_cfg bytes) and its batches, for a workspace at
// device address `ws`.  Every write into `img` is checked against the plan's
// region bounds before it is made.  allow_streams = false runs everything on
// one stream: a bulk lane plan level by level (its resident layout serves that
// order too), hoisted preps in their own slot (their blocks have memory of
// their own either way).
template <typename KeyT>
pase_status build_image(pase_graph_t g, char *ws, char *img, SearchImage &si, bool allow_streams = true);

}  // namespace pase

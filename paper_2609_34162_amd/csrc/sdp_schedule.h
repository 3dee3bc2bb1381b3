// Step-time model of the library's chunked schedules (streamed mode, its
// staged variant, the host-update route).  Plain C++, host only; compiled by
// the host compiler.  Not installed; not part of the ABI.
//
// The paper predicts a step from two quantities (Design, step-time model):
// a resource-demand lower bound, max over resources j of W_j / beta_j, and a
// dependency recurrence f(v) = d_v + max({a_v} and f(u) over the
// predecessors u of v), whose predecessors are data and version dependences,
// stream order and buffer release.  This model builds that graph for one
// call of the library, node for node as the runtime issues its work:
// copies, kernels and host-thread tasks on their streams, with the events
// the runtime records and waits on as the cross-stream edges.  Copy
// durations come from a fluid model of the host link: a copy moves at its
// direction's rate while it is alone on the link, and at its share of the
// bidirectional rate while the other direction is busy.  Host-thread tasks
// share host memory with the DMA: every byte a copy moves is read from or
// written to host memory, so the copies together move at most host_gbs, and
// while they run at a combined rate r a host task moves at most
// (host_gbs - dma_host_cost * r), and never more than its own peak.  A host
// thread that waits for a GPU command starts sync_us after the command's
// end.  With no overlap of copies in both directions and no copy beside a
// host task, the evaluation is exactly the recurrence with fixed durations.
#pragma once

#include <stdint.h>

#include <vector>

namespace sdp_sched {

struct Rates {
    double h2d_gbs, d2h_gbs, both_gbs;  // link: each direction alone; both at once (sum)
    double copy_cmd_us;                 // fixed cost of one copy command
    double norm_gbs;                    // norm pass and mean-gradient kernel (HBM bytes / s / 1e9)
    double update_gbs;                  // fused update kernel
    double launch_us;                   // fixed cost of one kernel
    double sync_us;                     // host round trip of the norm read-back
    double host_gbs;                    // host memory bandwidth of the host threads' copies
    double host_task_us;                // fixed cost of one hand-off to the host threads
    double host_adam_gbs;               // host AdamW lane alone (bytes read + written)
    double dep_us;                      // an event recorded on one GPU stream, waited on by the other
    double dma_host_cost;               // host memory bytes a host task loses per DMA byte
    double host_issue_us;               // host route: enqueueing one piece's kernel and copy
};

enum Schedule { kStreamed = 0, kStreamedStaged = 1, kHostRouteF32 = 2, kHostRouteBf16 = 3 };

struct Prediction {
    double predicted_ms;
    double bound_ms;
    double h2d_ms, d2h_ms, link_ms, gpu_ms, host_ms, dram_ms;
    int64_t n_chunks;
};

// The host-update route's pieces, in order: each segment is cut into
// consecutive pieces of at most `chunk` elements.  The piece size starts at
// chunk/16 (in whole multiples of kRampAlign; at `chunk` when chunk/16 is
// smaller than kRampAlign) and grows by 6/5, rounded up to a multiple of
// kRampAlign, after every piece until it reaches `chunk`; a piece that meets
// its segment's end is cut there.  The host threads then start after a short
// first copy, and each copy hides behind the host update of the piece before
// it while a copy takes at most 5/6 of the update's time per element.
constexpr int64_t kRampAlign = 65536;
struct RoutePiece {
    int32_t seg;
    int64_t off, len;
};
std::vector<RoutePiece> route_pieces(const std::vector<int64_t> &numels, int64_t chunk);

// Streamed mode's first pass moves only the R BF16 gradient arrays.  From
// pinned memory its chunks fill the staging slot that the update pass lays
// out for `chunk` elements: the largest multiple of the 65,536-element norm
// tile whose R arrays fit in (14 + 2R) * chunk bytes (at least `chunk`), so
// fewer, larger copies.  Staged, they keep `chunk`: the host threads fill a
// whole chunk's bounce buffer before its copy can start, and a larger first
// chunk holds the link back for longer.  The norm does not depend on the
// chunking.
inline int64_t norm_phase_chunk(int64_t chunk, int R, bool staged) {
    constexpr int64_t kTile = 65536;
    if (staged || chunk > INT64_MAX / (14 + 2 * (int64_t)R)) return chunk;
    const int64_t c = (14 + 2 * (int64_t)R) * chunk / (2 * (int64_t)R) / kTile * kTile;
    return c > chunk ? c : chunk;
}

// store_gbar: streamed mode keeps the mean gradient in device memory
// between its passes (the default) instead of streaming the gradients twice.
// host_cast: streamed mode rounds the BF16 parameters on the host from the
// returned master (12 B per element back instead of 14, and a host rounding
// task per chunk once its copies have landed).
Prediction predict(int schedule, const std::vector<int64_t> &numels, int R, int64_t chunk, bool store_gbar,
                   bool host_cast, const Rates &r);

}  // namespace sdp_sched

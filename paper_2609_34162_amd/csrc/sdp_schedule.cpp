// Step-time model of the chunked schedules; see sdp_schedule.h.
//
// The graph mirrors the runtime's issue order:
//  - streamed mode, phase 1: per chunk k (slot k mod 2; chunks of
//    norm_phase_chunk elements) the R gradient copies on the copy stream,
//    after the slot's previous norm kernel
//    (slot_free); the norm kernel on the compute stream after the copies
//    (h2d_done); then the finalize and the host's read-back of the norm;
//  - phase 2: per chunk, the state copies in after the slot's previous
//    outgoing copy, the update kernel, and the outgoing copies on the
//    compute stream, all issued after the read-back;
//  - staged variant: host-thread copies into pinned bounce buffer k mod 3
//    before each incoming copy (after that buffer's previous copy left it);
//    in phase 2 chunk j's results land in outgoing buffer j mod 3, and the
//    host thread stages and issues chunk j+2 before it drains chunk j, all
//    in the host thread's own order;
//  - host rounding of the BF16 parameters (either variant): 12 B per
//    element back, and after chunk j's copies land a host task reads its
//    master and writes its BF16 parameters, in the same issue order;
//  - host-update route: the norm pass and read-back, then per piece (see
//    route_pieces: a ramp of growing pieces, then chunks) the mean-gradient kernel
//    (after the slot's previous outgoing copy, and enqueued by the host
//    thread, which takes host_issue_us for it, after it finished the update
//    of piece j-2), its copy to the host on the copy stream, and the host
//    update after the copy.
#include "sdp_schedule.h"

#include <algorithm>
#include <cmath>
#include <limits>

namespace sdp_sched {
namespace {

enum Stream { kCopyS = 0, kCompS = 1, kHostS = 2, kStreams = 3 };
enum Kind { kFixed = 0, kH2D = 1, kD2H = 2, kHostWork = 3 };

struct Node {
    int stream = 0, kind = kFixed;
    double dur_us = 0.0;  // kFixed; kHostWork: the fixed hand-off cost before its bytes
    double bytes = 0.0;   // copies and host work
    double peak = 0.0;    // kHostWork: its own rate alone (bytes per us)
    int cmds = 0;         // copies: commands, each paying the fixed command cost
    std::vector<int> preds;
    int state = 0;  // 0 waiting, 1 command latency, 2 running / transferring, 3 done
    double t_end = 0.0, lat_end = 0.0, remaining = 0.0;
};

struct Graph {
    std::vector<Node> nodes;
    std::vector<int> fifo[kStreams];
    double h2d_bytes = 0.0, d2h_bytes = 0.0, gpu_us = 0.0, host_us = 0.0, host_bytes = 0.0;

    int add(int stream, int kind, double dur_us, double bytes, int cmds, std::initializer_list<int> preds) {
        Node n;
        n.stream = stream;
        n.kind = kind;
        n.dur_us = dur_us;
        n.bytes = bytes;
        n.cmds = cmds;
        for (int u : preds)
            if (u >= 0) n.preds.push_back(u);
        nodes.push_back(n);
        const int id = (int)nodes.size() - 1;
        fifo[stream].push_back(id);
        if (kind == kH2D) h2d_bytes += bytes;
        if (kind == kD2H) d2h_bytes += bytes;
        if (kind == kFixed && stream == kCompS) gpu_us += dur_us;
        if (kind == kFixed && stream == kHostS) host_us += dur_us;
        return id;
    }

    // A host-thread task: a hand-off cost, then `bytes` at up to `gbs`.
    int host(double bytes, double gbs, double task_us, std::initializer_list<int> preds) {
        const int id = add(kHostS, kHostWork, task_us, bytes, 0, preds);
        nodes[id].peak = gbs * 1e3;
        host_us += task_us + bytes / (gbs * 1e3);
        host_bytes += bytes;
        return id;
    }
};

// Finish time (us) of the graph: each stream runs its nodes in order, a node
// starts once its stream is free and its predecessors are done, and copies
// share the link as described in the header.
double evaluate(Graph &g, const Rates &r) {
    const size_t total = g.nodes.size();
    size_t head[kStreams] = {0, 0, 0};
    int cur[kStreams] = {-1, -1, -1};
    size_t done = 0;
    double t = 0.0;
    const double h2d = r.h2d_gbs * 1e3, d2h = r.d2h_gbs * 1e3, both = r.both_gbs * 1e3;  // bytes per us
    const double inf = std::numeric_limits<double>::infinity();
    // an edge between the copy and the compute stream is an event that one
    // queue records and the other waits on: it takes effect dep_us later; a
    // host thread waiting on a GPU command learns of its end sync_us later
    // (the round trip of the norm read-back)
    auto crosses = [](const Node &u, const Node &v) {
        return u.stream != v.stream && u.stream != kHostS && v.stream != kHostS;
    };
    auto wakes = [](const Node &u, const Node &v) { return u.stream != kHostS && v.stream == kHostS; };
    while (done < total) {
        double wake = inf;  // earliest time a node whose predecessors are done may start
        for (int s = 0; s < kStreams; ++s) {
            if (cur[s] >= 0 || head[s] >= g.fifo[s].size()) continue;
            const int id = g.fifo[s][head[s]];
            Node &v = g.nodes[id];
            bool ready = true;
            double at = t;
            for (int u : v.preds) {
                const Node &pu = g.nodes[u];
                if (pu.state != 3) {
                    ready = false;
                    break;
                }
                if (crosses(pu, v)) at = std::max(at, pu.t_end + r.dep_us);
                if (wakes(pu, v)) at = std::max(at, pu.t_end + r.sync_us);
            }
            if (!ready) continue;
            if (at > t) {
                wake = std::min(wake, at);
                continue;
            }
            cur[s] = id;
            if (v.kind == kFixed) {
                v.state = 2;
                v.t_end = t + v.dur_us;
            } else {
                v.state = 1;
                v.lat_end = t + (v.kind == kHostWork ? v.dur_us : v.cmds * r.copy_cmd_us);
                v.remaining = v.bytes;
            }
        }
        int nh = 0, nd = 0, nw = 0;
        for (int s = 0; s < kStreams; ++s) {
            if (cur[s] < 0) continue;
            const Node &v = g.nodes[cur[s]];
            if (v.state == 2 && v.kind == kH2D) ++nh;
            if (v.state == 2 && v.kind == kD2H) ++nd;
            if (v.state == 2 && v.kind == kHostWork) ++nw;
        }
        double rh = 0.0, rd = 0.0;
        if (nh && nd) {
            rh = std::min(h2d, both * h2d / (h2d + d2h));
            rd = std::min(d2h, both - rh);
        } else if (nh) {
            rh = h2d;
        } else if (nd) {
            rd = d2h;
        }
        // every DMA byte passes through host memory; the host threads get
        // what the copies leave of it, each DMA byte costing them
        // dma_host_cost bytes of host bandwidth
        const double dram = r.host_gbs * 1e3;
        if (rh + rd > dram) {
            const double f = dram / (rh + rd);
            rh *= f;
            rd *= f;
        }
        const double left = std::max(0.0, dram - r.dma_host_cost * (rh + rd));
        auto rate = [&](const Node &v) {
            if (v.kind == kH2D) return rh / nh;
            if (v.kind == kD2H) return rd / nd;
            return std::min(v.peak, left / nw);
        };
        double next = inf;
        int first = -1;
        for (int s = 0; s < kStreams; ++s) {
            if (cur[s] < 0) continue;
            const Node &v = g.nodes[cur[s]];
            double e;
            if (v.state == 1) e = v.lat_end;
            else if (v.kind == kFixed) e = v.t_end;
            else e = t + v.remaining / rate(v);
            if (e < next) {
                next = e;
                first = s;
            }
        }
        if (wake < next) {
            next = wake;
            first = -1;
        }
        if (next == inf) return std::numeric_limits<double>::quiet_NaN();  // nothing can run: not a valid schedule
        const double dt = next - t;
        for (int s = 0; s < kStreams; ++s) {
            if (cur[s] < 0) continue;
            Node &v = g.nodes[cur[s]];
            if (v.state == 2 && v.kind != kFixed) v.remaining -= rate(v) * dt;
        }
        if (first >= 0) {
            Node &v = g.nodes[cur[first]];
            if (v.state == 2 && v.kind != kFixed) v.remaining = 0.0;
        }
        t = next;
        for (int s = 0; s < kStreams; ++s) {
            if (cur[s] < 0) continue;
            Node &v = g.nodes[cur[s]];
            if (v.state == 1 && v.lat_end <= t) v.state = 2;
            bool fin = false;
            if (v.state == 2) {
                if (v.kind == kFixed) fin = v.t_end <= t;
                else fin = v.remaining <= 1e-9 * std::max(1.0, v.bytes);
            }
            if (fin) {
                v.state = 3;
                v.t_end = t;
                cur[s] = -1;
                ++head[s];
                ++done;
            }
        }
    }
    return t;
}

struct Chunk {
    int64_t len;
    bool full;  // len == chunk: the slot's arrays are back to back, so copies merge into one run
};

std::vector<Chunk> chunks_of(const std::vector<int64_t> &numels, int64_t C) {
    std::vector<Chunk> out;
    for (int64_t n : numels)
        for (int64_t off = 0; off < n; off += C) {
            const int64_t len = std::min(C, n - off);
            out.push_back({len, len == C});
        }
    return out;
}

double kernel_us(double bytes, double gbs, const Rates &r) { return bytes / (gbs * 1e3) + r.launch_us; }

}  // namespace

std::vector<RoutePiece> route_pieces(const std::vector<int64_t> &numels, int64_t chunk) {
    std::vector<RoutePiece> out;
    int64_t size = chunk / 16 / kRampAlign * kRampAlign;
    if (size < kRampAlign) size = chunk;
    for (size_t s = 0; s < numels.size(); ++s) {
        for (int64_t off = 0; off < numels[s];) {
            const int64_t len = std::min(size, numels[s] - off);
            out.push_back({(int32_t)s, off, len});
            off += len;
            if (size < chunk) {
                // size * 6/5 rounded down, then up to a whole kRampAlign; chunk
                // is a multiple of kRampAlign, so a size within one of it is chunk
                const int64_t grown = size + size / 5;
                size = grown > chunk - kRampAlign ? chunk : (grown + kRampAlign - 1) / kRampAlign * kRampAlign;
            }
        }
    }
    return out;
}

namespace {

// The staged runtime's bounce buffers and how far ahead its host thread
// stages (incoming buffers, outgoing buffers, chunks staged ahead of the
// drain), and the largest device-to-host copy it moves with its own kernel
// (one launch for all of a chunk's copies that qualify).
constexpr int kInBufs = 3, kOutBufs = 3, kStageAhead = 2;
constexpr double kD2HKernelMaxBytes = 64.0 * 1024 * 1024;

// Commands that carry one chunk's device-to-host copies of `sizes` bytes:
// one per copy above the kernel's limit, plus one launch for the rest.
int d2h_commands(const std::vector<double> &sizes, bool all_kernel) {
    int cmds = 0;
    bool launch = false;
    for (double b : sizes) {
        if (all_kernel || b <= kD2HKernelMaxBytes) launch = true;
        else ++cmds;
    }
    return cmds + (launch ? 1 : 0);
}

void build_streamed(Graph &g, const std::vector<int64_t> &numels, int R, int64_t C, bool store, bool staged,
                    bool host_cast, const Rates &r) {
    const std::vector<Chunk> ch1 = chunks_of(numels, norm_phase_chunk(C, R, staged));
    int slot_free[2] = {-1, -1}, bin_h2d[kInBufs] = {-1, -1, -1};
    for (size_t k = 0; k < ch1.size(); ++k) {
        const int sl = (int)(k & 1), bi = (int)(k % kInBufs);
        const double len = (double)ch1[k].len;
        int hin = -1;
        if (staged) hin = g.host(2.0 * 2 * R * len, r.host_gbs, r.host_task_us, {bin_h2d[bi]});
        const int cmds = (staged && ch1[k].full) ? 1 : R;
        const int h2d = g.add(kCopyS, kH2D, 0, 2.0 * R * len, cmds, {slot_free[sl], hin});
        const int norm = g.add(kCompS, kFixed, kernel_us((2.0 * R + (store ? 4.0 : 0.0)) * len, r.norm_gbs, r), 0, 0,
                               {h2d});
        slot_free[sl] = norm;
        bin_h2d[bi] = h2d;
    }
    const int fin = g.add(kCompS, kFixed, r.launch_us, 0, 0, {});
    const int rb = g.add(kHostS, kFixed, 0.0, 0, 0, {fin});  // the wake edge carries sync_us
    const size_t k0 = ch1.size();
    const std::vector<Chunk> ch = chunks_of(numels, C);
    int d2h_slot[2] = {-1, -1};
    std::vector<int> d2h_of(ch.size(), -1), drain_of(ch.size(), -1);
    const double in_bpe = 12.0 + (store ? 0.0 : 2.0 * R);
    const double out_bpe = host_cast ? 12.0 : 14.0;
    const bool ahead = staged || host_cast;  // the host waits for each chunk's results
    auto issue = [&](size_t j) {
        const int sl = (int)((j + k0) & 1), bi = (int)((j + k0) % kInBufs);
        const double len = (double)ch[j].len;
        int hin = -1;
        if (staged) hin = g.host(2.0 * in_bpe * len, r.host_gbs, r.host_task_us, {rb, bin_h2d[bi]});
        const int in_cmds = (staged && ch[j].full) ? 1 : 3 + (store ? 0 : R);
        const int h2d = g.add(kCopyS, kH2D, 0, in_bpe * len, in_cmds, {rb, hin, d2h_slot[sl]});
        const int upd = g.add(kCompS, kFixed, kernel_us((26.0 + (store ? 4.0 : 2.0 * R)) * len, r.update_gbs, r), 0,
                              0, {h2d, rb});
        // master, m and v, and the BF16 parameters unless the host rounds them;
        // staged, a full chunk's arrays sit back to back and leave as one run
        std::vector<double> sizes = {4.0 * len, 4.0 * len, 4.0 * len};
        if (!host_cast) sizes.push_back(2.0 * len);
        if (staged && ch[j].full) sizes = {out_bpe * len};
        const int out_cmds = d2h_commands(sizes, host_cast && !staged);
        const int buf_free = (ahead && j >= (size_t)kOutBufs) ? drain_of[j - kOutBufs] : -1;
        d2h_of[j] = g.add(kCompS, kD2H, 0, out_bpe * len, out_cmds, {upd, hin, buf_free});
        bin_h2d[bi] = h2d;
        d2h_slot[sl] = d2h_of[j];
    };
    if (!ahead) {
        for (size_t j = 0; j < ch.size(); ++j) issue(j);
        return;
    }
    size_t next = 0;
    for (size_t j = 0; j < ch.size(); ++j) {
        for (; next < ch.size() && next <= j + kStageAhead; ++next) issue(next);
        // staged: the results move out of the bounce buffer (read and
        // written); host rounding: the master read, the BF16 parameters written
        const double len = (double)ch[j].len;
        const double bytes = (staged ? 2.0 * out_bpe * len : 0.0) + (host_cast ? 6.0 * len : 0.0);
        drain_of[j] = g.host(bytes, r.host_gbs, r.host_task_us, {d2h_of[j]});
    }
}

void build_host_route(Graph &g, const std::vector<int64_t> &numels, int R, int64_t C, bool bf16, const Rates &r) {
    for (int64_t n : numels) g.add(kCompS, kFixed, kernel_us(2.0 * R * (double)n, r.norm_gbs, r), 0, 0, {});
    const int fin = g.add(kCompS, kFixed, r.launch_us, 0, 0, {});
    const int rb = g.add(kHostS, kFixed, 0.0, 0, 0, {fin});  // the wake edge carries sync_us
    std::vector<Chunk> ch;
    for (const RoutePiece &pc : route_pieces(numels, C)) ch.push_back({pc.len, false});
    const double esz = bf16 ? 2.0 : 4.0;
    std::vector<int> d2h(ch.size(), -1), adam(ch.size(), -1);
    auto issue = [&](size_t j, int host_pred) {
        const double len = (double)ch[j].len;
        const int slot_pred = j >= 2 ? d2h[j - 2] : -1;
        const int gk = g.add(kCompS, kFixed, kernel_us((2.0 * R + esz) * len, r.norm_gbs, r), 0, 0,
                             {rb, host_pred, slot_pred});
        d2h[j] = g.add(kCopyS, kD2H, 0, esz * len, 1, {gk});
    };
    if (!ch.empty()) issue(0, -1);
    for (size_t j = 0; j < ch.size(); ++j) {
        // the calling thread enqueues the next piece, then waits for this
        // piece's copy and updates it
        if (j + 1 < ch.size()) issue(j + 1, g.add(kHostS, kFixed, r.host_issue_us, 0, 0, {}));
        adam[j] = g.host((26.0 + esz) * (double)ch[j].len, r.host_adam_gbs, r.host_task_us, {d2h[j]});
    }
}

}  // namespace

Prediction predict(int schedule, const std::vector<int64_t> &numels, int R, int64_t chunk, bool store_gbar,
                   bool host_cast, const Rates &r) {
    Graph g;
    if (schedule == kStreamed || schedule == kStreamedStaged)
        build_streamed(g, numels, R, chunk, store_gbar, schedule == kStreamedStaged, host_cast, r);
    else
        build_host_route(g, numels, R, chunk, schedule == kHostRouteBf16, r);
    Prediction p{};
    for (int64_t n : numels) p.n_chunks += n / chunk + (n % chunk != 0);  // no overflow near the int64 limit
    p.h2d_ms = g.h2d_bytes / (r.h2d_gbs * 1e9) * 1e3;
    p.d2h_ms = g.d2h_bytes / (r.d2h_gbs * 1e9) * 1e3;
    p.link_ms = (g.h2d_bytes + g.d2h_bytes) / (r.both_gbs * 1e9) * 1e3;
    p.gpu_ms = g.gpu_us / 1e3;
    p.host_ms = g.host_us / 1e3;
    // host memory carries the host tasks' bytes and every DMA byte
    p.dram_ms = (g.host_bytes + g.h2d_bytes + g.d2h_bytes) / (r.host_gbs * 1e9) * 1e3;
    p.bound_ms = std::max({p.h2d_ms, p.d2h_ms, p.link_ms, p.gpu_ms, p.host_ms, p.dram_ms});
    p.predicted_ms = evaluate(g, r) / 1e3;
    return p;
}

}  // namespace sdp_sched

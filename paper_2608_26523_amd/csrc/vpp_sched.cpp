// Discrete-event model of CPP / VPP / VPP-Async / pipelined packing on two
// pipeline ranks (sections 2.4, 5.1-5.3). The interface and the model are
// described in vpp_sched.h.
//
// Each rank executes a program: per request, a list of items, each either a
// compute operation or a synchronous transfer (a rendezvous of both ranks).
// The simulation advances over the distinct event times. At each time every
// free rank, rank 0 first, starts its next item if that item is ready, and
// this repeats until no rank starts anything more at that time (a zero-length
// item or a rendezvous can make the other rank's item ready at the same time).
#include "vpp_sched.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <new>
#include <queue>
#include <vector>

namespace {

constexpr double NEVER = std::numeric_limits<double>::infinity();

struct Op {
    int32_t req, chunk, stage, rank;
    double dur;
    int pred_stage;  // (req, chunk, stage-1) or -1
    int pred_chunk;  // (req, chunk-1, stage) or -1
    bool cross;      // pred_stage ran on the other rank
    double start = -1.0, end = -1.0;
};

// A synchronous transfer: both ranks take part; each records the chunk it sends.
struct Xfer {
    int32_t req;
    int32_t sent[2] = {-1, -1};
    bool at[2] = {false, false};  // rank has reached it (and waits there)
    double start = -1.0;
};

struct Item {
    bool xfer;
    int idx;  // op index or transfer index
};

struct Model {
    const vpp_sched_problem_t& p;
    std::vector<Op> ops;
    std::vector<Xfer> xfers;
    std::vector<std::vector<Item>> prog[2];  // prog[rank][request]
    std::vector<int> base;                   // first op index of each request

    explicit Model(const vpp_sched_problem_t& pr) : p(pr) {}

    int nstages() const { return p.layout == VPP_LAYOUT_CPP ? 2 : 4; }
    static int rank_of(int layout, int stage) {
        if (layout == VPP_LAYOUT_CPP) return stage;
        return (stage == 1 || stage == 2) ? 1 : 0;  // fold-back: s0, s3 on rank 0
    }
    int op_index(int r, int k, int s) const { return base[r] + k * nstages() + s; }

    void build_ops() {
        const int S = nstages();
        int64_t t = 0;
        base.resize(p.num_requests);
        for (int r = 0; r < p.num_requests; ++r) {
            base[r] = (int)ops.size();
            for (int k = 0; k < p.num_chunks[r]; ++k, ++t) {
                const double tau = p.stage_time[t];
                for (int s = 0; s < S; ++s) {
                    Op o;
                    o.req = r;
                    o.chunk = k;
                    o.stage = s;
                    o.rank = rank_of(p.layout, s);
                    o.dur = p.layout == VPP_LAYOUT_CPP ? tau + tau : tau;
                    o.pred_stage = s > 0 ? base[r] + k * S + s - 1 : -1;
                    o.pred_chunk = k > 0 ? base[r] + (k - 1) * S + s : -1;
                    o.cross = s > 0 && rank_of(p.layout, s - 1) != o.rank;
                    ops.push_back(o);
                }
            }
        }
    }

    int new_xfer(int r) {
        Xfer x;
        x.req = r;
        xfers.push_back(x);
        return (int)xfers.size() - 1;
    }
    void push_op(int rank, int r, int op) { prog[rank][r].push_back({false, op}); }
    void push_xfer(int rank, int r, int x) { prog[rank][r].push_back({true, x}); }

    void build_programs() {
        const bool sync = p.comm == VPP_COMM_SYNC;
        for (int rank = 0; rank < 2; ++rank) prog[rank].assign(p.num_requests, {});
        for (int r = 0; r < p.num_requests; ++r) {
            const int N = p.num_chunks[r];
            if (p.layout == VPP_LAYOUT_CPP) {
                for (int k = 0; k < N; ++k) {
                    push_op(0, r, op_index(r, k, 0));
                    if (sync) {
                        const int x = new_xfer(r);
                        xfers[x].sent[0] = k;
                        push_xfer(0, r, x);
                        push_xfer(1, r, x);
                    }
                    push_op(1, r, op_index(r, k, 1));
                }
                continue;
            }
            // VPP. Transfer j (sync mode) carries chunk j forward and chunk j-1
            // back: j = 0 forward only, j = N back only (chunk N-1).
            std::vector<int> x(N + 1, -1);
            if (sync)
                for (int j = 0; j <= N; ++j) {
                    x[j] = new_xfer(r);
                    xfers[x[j]].sent[0] = j < N ? j : -1;
                    xfers[x[j]].sent[1] = j > 0 ? j - 1 : -1;
                }
            // rank 1: s1, s2 of each chunk, with the transfers around them
            for (int k = 0; k < N; ++k) {
                if (sync && k == 0) push_xfer(1, r, x[0]);
                push_op(1, r, op_index(r, k, 1));
                push_op(1, r, op_index(r, k, 2));
                if (sync) push_xfer(1, r, x[k + 1]);
            }
            // rank 0: s0 of chunks 0 and 1, then per period k = 1 .. N-1 the exit
            // s3 of chunk k-1 and the entry s0 of chunk k+1, then s3 of chunk N-1
            push_op(0, r, op_index(r, 0, 0));
            if (sync) push_xfer(0, r, x[0]);
            if (N > 1) {
                push_op(0, r, op_index(r, 1, 0));
                if (sync) push_xfer(0, r, x[1]);
            }
            for (int k = 1; k < N; ++k) {
                const int exit_op = op_index(r, k - 1, 3);
                const bool has_entry = k + 1 < N;
                if (has_entry && p.entry_first) {
                    push_op(0, r, op_index(r, k + 1, 0));
                    push_op(0, r, exit_op);
                } else {
                    push_op(0, r, exit_op);
                    if (has_entry) push_op(0, r, op_index(r, k + 1, 0));
                }
                if (sync) push_xfer(0, r, x[k + 1]);
            }
            if (sync && N == 1) push_xfer(0, r, x[1]);  // the only chunk's back transfer
            push_op(0, r, op_index(r, N - 1, 3));
        }
    }

    // time at which op o's inputs are all available (NEVER if a predecessor has not finished)
    double inputs_ready(const Op& o) const {
        double t = 0.0;
        if (o.pred_chunk >= 0) {
            const Op& q = ops[o.pred_chunk];
            if (q.end < 0) return NEVER;
            t = std::max(t, q.end);
        }
        if (o.pred_stage >= 0) {
            const Op& q = ops[o.pred_stage];
            if (q.end < 0) return NEVER;
            const double arrive = (o.cross && p.comm == VPP_COMM_ASYNC) ? q.end + p.comm_time : q.end;
            t = std::max(t, arrive);
        }
        return t;
    }
};

bool valid(const vpp_sched_problem_t* p) {
    if (!p) return false;
    if (p->layout != VPP_LAYOUT_CPP && p->layout != VPP_LAYOUT_VPP) return false;
    if (p->comm != VPP_COMM_SYNC && p->comm != VPP_COMM_ASYNC) return false;
    if ((p->entry_first != 0 && p->entry_first != 1) || (p->packing != 0 && p->packing != 1)) return false;
    if (p->packing && p->comm != VPP_COMM_ASYNC) return false;
    if (p->num_requests < 1 || !p->num_chunks || !p->stage_time) return false;
    if (!(p->comm_time >= 0.0) || !std::isfinite(p->comm_time)) return false;
    int64_t total = 0;
    for (int r = 0; r < p->num_requests; ++r) {
        if (p->num_chunks[r] < 1) return false;
        total += p->num_chunks[r];
        if (total > (int64_t)1 << 20) return false;
    }
    for (int64_t i = 0; i < total; ++i)
        if (!(p->stage_time[i] >= 0.0) || !std::isfinite(p->stage_time[i])) return false;
    return true;
}

int64_t count_events(const vpp_sched_problem_t* p) {
    int64_t n = 0;
    for (int r = 0; r < p->num_requests; ++r) {
        const int64_t N = p->num_chunks[r];
        if (p->layout == VPP_LAYOUT_CPP) n += 2 * N + (p->comm == VPP_COMM_SYNC ? 2 * N : 0);
        else n += 4 * N + (p->comm == VPP_COMM_SYNC ? 2 * (N + 1) : 0);
    }
    return n;
}

vpp_status_t run(const vpp_sched_problem_t& pr, vpp_sched_summary_t* sum, double* request_end,
                 vpp_sched_event_t* events, int64_t cap) {
    Model m(pr);
    m.build_ops();
    m.build_programs();
    const int R = pr.num_requests;
    std::vector<size_t> head[2] = {std::vector<size_t>(R, 0), std::vector<size_t>(R, 0)};
    double free_at[2] = {0.0, 0.0};   // the rank is busy until then
    double compute[2] = {0.0, 0.0}, exposed[2] = {0.0, 0.0};
    std::priority_queue<double, std::vector<double>, std::greater<double>> times;
    size_t remaining = 0;
    for (int rank = 0; rank < 2; ++rank)
        for (int r = 0; r < R; ++r) remaining += m.prog[rank][r].size();

    // the request whose head this rank considers first, and whether later ones may run
    auto first_open = [&](int rank) {
        for (int r = 0; r < R; ++r)
            if (head[rank][r] < m.prog[rank][r].size()) return r;
        return R;
    };
    // try to start one item on a free rank at time T; true if something started
    auto try_start = [&](int rank, double T) -> bool {
        if (free_at[rank] > T) return false;
        const int r0 = first_open(rank);
        const int r_last = pr.packing ? R - 1 : r0;
        for (int r = r0; r <= r_last && r < R; ++r) {
            if (head[rank][r] >= m.prog[rank][r].size()) continue;
            const Item it = m.prog[rank][r][head[rank][r]];
            if (it.xfer) {
                Xfer& x = m.xfers[it.idx];
                if (!x.at[rank]) x.at[rank] = true;
                const int other = 1 - rank;
                if (!x.at[other]) continue;  // waits for the peer (sync mode: no packing)
                x.start = T;
                const double end = T + pr.comm_time;
                for (int q = 0; q < 2; ++q) {
                    free_at[q] = end;
                    exposed[q] += pr.comm_time;
                    ++head[q][r];
                    --remaining;
                }
                times.push(end);
                return true;
            }
            Op& o = m.ops[it.idx];
            const double ready = m.inputs_ready(o);
            if (ready > T) continue;
            // exposed communication: idle that only the transfer's flight time caused
            if (o.cross && pr.comm == VPP_COMM_ASYNC && o.pred_stage >= 0) {
                double no_comm = std::max(free_at[rank], m.ops[o.pred_stage].end);
                if (o.pred_chunk >= 0) no_comm = std::max(no_comm, m.ops[o.pred_chunk].end);
                if (T > no_comm) exposed[rank] += T - no_comm;
            }
            o.start = T;
            o.end = T + o.dur;
            free_at[rank] = o.end;
            compute[rank] += o.dur;
            ++head[rank][r];
            --remaining;
            times.push(o.end);
            return true;
        }
        return false;
    };
    // future time at which a waiting head may become ready (message arrivals)
    auto push_arrivals = [&](double T) {
        for (int rank = 0; rank < 2; ++rank)
            for (int r = 0; r < R; ++r) {
                if (head[rank][r] >= m.prog[rank][r].size()) continue;
                const Item it = m.prog[rank][r][head[rank][r]];
                if (it.xfer) continue;
                const double ready = m.inputs_ready(m.ops[it.idx]);
                if (ready > T && ready < NEVER) times.push(ready);
            }
    };

    double T = 0.0;
    times.push(0.0);
    while (remaining > 0) {
        if (times.empty()) return VPP_ERR_INVALID_ARG;  // no progress possible (cannot happen for valid programs)
        T = times.top();
        while (!times.empty() && times.top() <= T) times.pop();
        bool any = true;
        while (any) {
            any = false;
            for (int rank = 0; rank < 2; ++rank)
                while (try_start(rank, T)) any = true;
        }
        push_arrivals(T);
        if (times.empty() && remaining > 0) {
            // nothing in flight: a free rank waits for a rank that is busy
            const double t_next = std::min(free_at[0] > T ? free_at[0] : NEVER, free_at[1] > T ? free_at[1] : NEVER);
            if (t_next == NEVER) return VPP_ERR_INVALID_ARG;
            times.push(t_next);
        }
    }

    double makespan = 0.0;
    for (const Op& o : m.ops) makespan = std::max(makespan, o.end);
    for (const Xfer& x : m.xfers) makespan = std::max(makespan, x.start + pr.comm_time);
    sum->makespan = makespan;
    for (int q = 0; q < 2; ++q) {
        sum->compute[q] = compute[q];
        sum->exposed_comm[q] = exposed[q];
        sum->idle[q] = makespan - compute[q] - exposed[q];
    }
    sum->bubble_ratio = makespan > 0.0 ? (sum->idle[0] + sum->idle[1]) / (2.0 * makespan) : 0.0;
    if (request_end) {
        for (int r = 0; r < R; ++r) request_end[r] = 0.0;
        for (const Op& o : m.ops) request_end[o.req] = std::max(request_end[o.req], o.end);
        for (const Xfer& x : m.xfers) request_end[x.req] = std::max(request_end[x.req], x.start + pr.comm_time);
    }
    if (events) {
        std::vector<vpp_sched_event_t> ev;
        ev.reserve(m.ops.size() + 2 * m.xfers.size());
        for (const Op& o : m.ops) ev.push_back({o.req, o.chunk, o.stage, o.rank, o.start, o.end});
        for (const Xfer& x : m.xfers)
            for (int q = 0; q < 2; ++q) ev.push_back({x.req, x.sent[q], -1, q, x.start, x.start + pr.comm_time});
        std::stable_sort(ev.begin(), ev.end(), [](const vpp_sched_event_t& a, const vpp_sched_event_t& b) {
            return a.start < b.start || (a.start == b.start && a.rank < b.rank);
        });
        if ((int64_t)ev.size() > cap) return VPP_ERR_INVALID_ARG;
        std::copy(ev.begin(), ev.end(), events);
    }
    return VPP_OK;
}

}  // namespace

extern "C" vpp_status_t vpp_sched_event_count(const vpp_sched_problem_t* problem, int64_t* count) {
    if (!count || !valid(problem)) return VPP_ERR_INVALID_ARG;
    *count = count_events(problem);
    return VPP_OK;
}

extern "C" vpp_status_t vpp_sched_simulate(const vpp_sched_problem_t* problem, vpp_sched_summary_t* summary,
                                           double* request_end, vpp_sched_event_t* events,
                                           int64_t events_capacity) {
    if (!summary || !valid(problem)) return VPP_ERR_INVALID_ARG;
    if (events && events_capacity < count_events(problem)) return VPP_ERR_INVALID_ARG;
    try {
        return run(*problem, summary, request_end, events, events_capacity);
    } catch (const std::bad_alloc&) {
        return VPP_ERR_NOMEM;
    }
}

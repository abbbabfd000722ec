// Layerwise pipeline (Section 3.5, eq. (3)) with a host producer standing in
// for the storage server's layerwise GET (Section 3.3 and the appendix
// pseudocode): for each layer, in prefix order, the producer copies that
// layer's slice of every matched chunk object into a pinned slot, paced to a
// byte rate, and then signals layer-ready.  The driver thread lands the slot
// in HBM with asynchronous DMAs on the copy stream -- from a paced in-order
// producer, span by span as the leading bytes of the slot complete, so the
// copy overlaps the production -- and, once the whole layer is in, ingests it;
// the compute stream waits on the layer's ingested event and runs that
// layer's attention.  So layer l+1 lands and is ingested while layer l
// computes, and every hand-off is a HIP event, never a device-wide sync.
//
// Slot reuse: the pinned slot of item k is refilled for item k+slots only
// after item k's DMA has completed (landed event); the HBM slot is reused
// in copy-stream order, after the ingest that read it.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <memory>
#include <mutex>
#include <queue>
#include <string>
#include <thread>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "common.hpp"

namespace oc {

using Clock = std::chrono::steady_clock;

struct Slot {
    void *pinned = nullptr;
    void *device = nullptr;
};

struct Context {
    int device = 0;
    oc_kv_pool pool{};
    oc_pipeline_opts opts{};
    int64_t max_prefix = 0, max_suffix = 0;
    size_t slot_bytes = 0;
    hipStream_t copy = nullptr, compute = nullptr;
    std::vector<hipStream_t> req_streams;   // per-request compute streams (emulated compute windows)
    std::vector<Slot> slots;
    void *ws = nullptr;                // attention workspace, one slice per stream in use
    size_t ws_bytes = 0;
    bool has_layer = false;            // rest-of-layer compute after each attention
    oc_layer_weights lw{};
    void *lbuf = nullptr;              // its stage buffers, one set per stream in use
    size_t lbuf_bytes = 0;
    std::vector<hipEvent_t> events;    // pool of timing events, reused across runs
    hipEvent_t caller_done = nullptr;  // null-stream work enqueued before a run
    double last_ms = 0.0;
};

// A roctx range for a scope of the calling thread (a no-op without a tool
// attached): the run and each layer's enqueue show on a rocprofv3 timeline.
struct TraceRange {
    explicit TraceRange(const std::string &name) { roctxRangePushA(name.c_str()); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange &) = delete;
    TraceRange &operator=(const TraceRange &) = delete;
};

// ---- shared state between the driver and the producer ----------------------
struct RunShared {
    std::mutex mu;
    std::condition_variable cv;
    int64_t ready = 0;            // items whose payload is complete in a pinned slot
    int64_t landed_recorded = 0;  // items whose landed event has been recorded
    bool abort = false;           // driver -> producer: stop now
    int producer_status = OC_OK;  // producer -> driver
    std::string producer_msg;
    std::deque<int64_t> reported; // rate producer -> driver: items complete in a pinned slot
    std::vector<int64_t> delivered; // per item: bytes the producer put in its pinned slot,
                                    // set before the item is published as ready or reported
    // producer -> driver, layerwise items of the in-order producer: the
    // leading bytes of item part_item's slot that are complete (whole
    // pieces, in slot order); never decreases for an item
    int64_t part_item = -1, part_bytes = 0;
};

// The injected short write: the copy of item `it`'s last chunk stops half
// way, as a torn read of an object would.  Returns the bytes to copy of a
// unit that is the `j`-th of [.., last).
static inline int64_t copy_len(const oc_pipeline_opts &o, int32_t layer, int64_t j, int64_t last, int64_t unit) {
    return o.fault == OC_FAULT_SHORT_WRITE && layer == o.fault_layer && j == last - 1 ? unit / 2 : unit;
}

// A layer payload of the in-order, rate-capped producer lands in HBM in spans
// of about this many bytes as its leading pieces complete: an eighth of the
// layer, at least 8 MiB and a piece.  Each copy costs the driver thread about
// 50 us, which must stay well below a span's time on the host link (8 MiB:
// about 150 us).  The producer wakes the driver only when a span boundary is
// passed.  Uncapped, the producer outruns the host link and each layer's DMA
// already overlaps the next layer's production: the layer lands whole.
static inline int64_t landing_span(const oc_pipeline_opts &o, int64_t layer_bytes) {
    if (!(o.rate_bytes_per_s > 0)) return std::max<int64_t>(layer_bytes, 1);
    return std::max<int64_t>({o.piece_bytes, layer_bytes / 8, (int64_t)8 << 20});
}

// Starts up to n threads running fn, fewer if the system refuses more;
// returns how many run.
template <class F>
static int start_threads(std::vector<std::thread> &pool, int n, F fn) {
    for (int i = 0; i < n; ++i) {
        try {
            pool.emplace_back(fn);
        } catch (...) {
            break;
        }
    }
    return (int)pool.size();
}

// Writes zeros over [p, p + bytes) from up to `threads` threads (the rest
// on the calling thread if the system refuses more), faulting every page in;
// a ring under 64 MiB per slot is written by the calling thread alone.
static void prefault(unsigned char *p, size_t bytes, int threads) {
    if (bytes < ((size_t)64 << 20) || threads <= 1) {
        std::memset(p, 0, bytes);
        return;
    }
    const size_t part = (bytes + (size_t)threads - 1) / (size_t)threads;
    std::vector<std::thread> pool;
    size_t done = 0;
    for (int i = 0; i < threads && done < bytes; ++i) {
        const size_t len = std::min(part, bytes - done);
        try {
            pool.emplace_back([p, done, len] { std::memset(p + done, 0, len); });
        } catch (...) {
            break;
        }
        done += len;
    }
    if (done < bytes) std::memset(p + done, 0, bytes - done);
    for (auto &t : pool) t.join();
}

// Stall and abort stop delivery at fault_layer; a short write still delivers.
static inline bool stops_at(const oc_pipeline_opts &o, int32_t layer) {
    return (o.fault == OC_FAULT_STALL || o.fault == OC_FAULT_ABORT) && layer == o.fault_layer;
}

// A unit of delivery: one layer payload of a request (layerwise), or a
// group of whole chunk objects j0..j1-1 of a request (chunkwise, layer 0 for
// the fault injection).
struct Item {
    int32_t layer;
    int32_t req;
    bool chunks = false;
    int64_t j0 = 0, j1 = 0;
};

static int fill_defaults(oc_pipeline_opts &o) {
    if (o.piece_bytes <= 0) o.piece_bytes = 1 << 20;
    if (o.slots <= 0) o.slots = 3;
    if (o.producer_threads <= 0) o.producer_threads = 4;
    if (o.timeout_ms <= 0) o.timeout_ms = 60000;
    if (o.slots < 2) return fail(OC_EINVAL, "at least 2 staging slots are needed");
    if (o.producer_threads > 64) return fail(OC_EINVAL, "producer_threads must be <= 64");
    if (o.mode < OC_MODE_HBM_RESIDENT || o.mode > OC_MODE_PRODUCER) return fail(OC_EINVAL, "unknown mode");
    if (o.rate_bytes_per_s < 0) return fail(OC_EINVAL, "negative rate");
    if (o.fault < OC_FAULT_NONE || o.fault > OC_FAULT_SHORT_WRITE) return fail(OC_EINVAL, "unknown fault");
    if (o.alloc_policy < OC_ALLOC_FIFO || o.alloc_policy > OC_ALLOC_CAL_STALL_OPT)
        return fail(OC_EINVAL, "unknown allocation policy");
    if (o.alloc_policy != OC_ALLOC_FIFO && !(o.rate_bytes_per_s > 0))
        return fail(OC_EINVAL, "an allocation policy needs a positive budget (rate_bytes_per_s)");
    if (o.margin_bytes_per_s < 0) return fail(OC_EINVAL, "negative margin");
    if (o.delivery < OC_DELIVERY_LAYERWISE || o.delivery > OC_DELIVERY_AUTO) return fail(OC_EINVAL, "unknown delivery");
    if (o.theta_bytes < 0) return fail(OC_EINVAL, "negative theta_bytes");
    if (o.delivery == OC_DELIVERY_CHUNKWISE && o.alloc_policy != OC_ALLOC_FIFO)
        return fail(OC_EINVAL, "allocation policies schedule layerwise requests; chunkwise delivery needs OC_ALLOC_FIFO");
    return OC_OK;
}

// Makes `dev` current for a scope and gives the caller back its own device.
struct DeviceScope {
    int prev = -1;
    explicit DeviceScope(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        (void)hipSetDevice(dev);
    }
    ~DeviceScope() {
        if (prev >= 0) hipSetDevice(prev);
    }
};

static void release(Context *c) {
    if (!c) return;
    const DeviceScope on_device(c->device);
    if (c->copy) hipStreamSynchronize(c->copy);
    if (c->compute) hipStreamSynchronize(c->compute);
    for (auto st : c->req_streams) hipStreamSynchronize(st);
    for (auto &s : c->slots) {
        if (s.pinned) hipHostFree(s.pinned);
        if (s.device) hipFree(s.device);
    }
    for (auto e : c->events) hipEventDestroy(e);
    if (c->caller_done) hipEventDestroy(c->caller_done);
    if (c->ws) hipFree(c->ws);
    if (c->lbuf) hipFree(c->lbuf);
    if (c->copy) hipStreamDestroy(c->copy);
    if (c->compute) {
        forget_blas_stream(c->compute);
        hipStreamDestroy(c->compute);
    }
    for (auto st : c->req_streams) {
        forget_blas_stream(st);
        hipStreamDestroy(st);
    }
    delete c;
}

// ---- producer -------------------------------------------------------------
// Copies item after item into pinned slots.  Pieces of an item go to a pool
// of worker threads; piece p of the run may start once the wall clock has
// reached  t0 + (bytes delivered before it + its own bytes) / rate.
struct Producer {
    Context *c;
    RunShared *sh;
    const oc_request *reqs;
    const std::vector<Item> *items;
    Clock::time_point t0;
    std::vector<double> *produced_ms;   // per item
    std::vector<hipEvent_t> *landed;    // per item
    double rate;
    int64_t S;                          // bytes per chunk slice
    int32_t L;

    // per-item work shared with the workers
    std::mutex wmu;
    std::condition_variable wcv;
    int64_t cur_item = -1, next_piece = 0, n_pieces = 0, pieces_done = 0, chunks_per_piece = 1;
    int64_t bytes_done = 0;             // bytes the current item's pieces copied
    std::vector<char> piece_done;       // per piece of the current item
    int64_t prefix_pieces = 0;          // leading pieces of the current item that are done
    double cum_before = 0.0;            // bytes delivered before the current item
    bool stop = false;

    bool aborted() {
        std::lock_guard<std::mutex> g(sh->mu);
        return sh->abort;
    }

    void worker() {
        for (;;) {
            int64_t item, p, cpp;
            double cum;
            {
                std::unique_lock<std::mutex> lk(wmu);
                wcv.wait(lk, [&] { return stop || (cur_item >= 0 && next_piece < n_pieces); });
                if (stop) return;
                item = cur_item;
                p = next_piece++;
                cpp = chunks_per_piece;
                cum = cum_before;
            }
            const Item it = (*items)[item];
            const oc_request &r = reqs[it.req];
            const int64_t N = r.prefix_tokens / c->pool.layout.chunk_tokens;
            // layerwise: layer `it.layer` of every chunk, S bytes each;
            // chunkwise: whole objects it.j0..it.j1-1, L*S bytes each
            const int64_t unit = it.chunks ? (int64_t)L * S : S;
            const int64_t first = it.chunks ? it.j0 : 0, last = it.chunks ? it.j1 : N;
            const int64_t src_off = it.chunks ? 0 : (int64_t)it.layer * S;
            const int64_t j0 = first + p * cpp, j1 = std::min(last, j0 + cpp);
            bool skip = false;
            if (rate > 0) {
                const double t_release = (cum + (double)(j1 - first) * unit) / rate;
                const auto when = t0 + std::chrono::duration_cast<Clock::duration>(std::chrono::duration<double>(t_release));
                // sleep most of the way in steps of at most 20 ms (a stopped
                // run ends the wait), then spin for a microsecond-accurate release
                for (;;) {
                    auto now = Clock::now();
                    if (now >= when) break;
                    auto left = when - now;
                    if (left > std::chrono::microseconds(200)) {
                        std::this_thread::sleep_for(std::min<Clock::duration>(left - std::chrono::microseconds(100),
                                                                             std::chrono::milliseconds(20)));
                        if (aborted()) {
                            skip = true;
                            break;
                        }
                    }
                }
            }
            unsigned char *dst = static_cast<unsigned char *>(c->slots[item % c->slots.size()].pinned);
            int64_t copied = 0;
            for (int64_t j = j0; j < j1 && !skip; ++j) {
                const unsigned char *obj = static_cast<const unsigned char *>(r.chunk_objects[j]);
                const int64_t len = copy_len(c->opts, it.layer, j, last, unit);
                std::memcpy(dst + (j - first) * unit, obj + src_off, (size_t)len);
                copied += len;
            }
            int64_t prefix = -1;      // complete leading bytes of a layer payload's slot
            {
                std::lock_guard<std::mutex> g(wmu);
                ++pieces_done;
                bytes_done += copied;
                if (!skip) {
                    piece_done[p] = 1;
                    while (prefix_pieces < n_pieces && piece_done[prefix_pieces]) ++prefix_pieces;
                    if (!it.chunks) prefix = std::min(prefix_pieces * cpp, last - first) * unit;
                }
            }
            wcv.notify_all();
            if (prefix >= 0) {
                const int64_t span = landing_span(c->opts, (last - first) * unit);
                bool wake = false;
                {
                    std::lock_guard<std::mutex> g(sh->mu);
                    if (item > sh->part_item || (item == sh->part_item && prefix > sh->part_bytes)) {
                        const int64_t before = item == sh->part_item ? sh->part_bytes : 0;
                        wake = prefix / span > before / span;
                        sh->part_item = item;
                        sh->part_bytes = prefix;
                    }
                }
                if (wake) sh->cv.notify_all();
            }
        }
    }

    void set_error(int st, const char *msg) {
        std::lock_guard<std::mutex> g(sh->mu);
        if (sh->producer_status == OC_OK) {
            sh->producer_status = st;
            sh->producer_msg = msg;
        }
        sh->cv.notify_all();
    }

    void run() {
        std::vector<std::thread> pool;
        if (start_threads(pool, c->opts.producer_threads, [this] { worker(); }) == 0) {
            set_error(OC_ENOMEM, "could not start the producer's copy threads");
            return;
        }
        double cum = 0.0;
        const int64_t n_items = (int64_t)items->size();
        const int64_t nslots = (int64_t)c->slots.size();
        for (int64_t k = 0; k < n_items; ++k) {
            const Item it = (*items)[k];
            if (stops_at(c->opts, it.layer)) {
                if (c->opts.fault == OC_FAULT_ABORT) {
                    set_error(OC_EABORT, "producer aborted (injected fault)");
                    break;
                }
                // injected stall: deliver nothing more until the driver gives up
                std::unique_lock<std::mutex> lk(sh->mu);
                sh->cv.wait(lk, [&] { return sh->abort; });
                break;
            }
            // the pinned slot is free once the DMA of item k - slots has landed
            if (k >= nslots) {
                const int64_t prev = k - nslots;
                std::unique_lock<std::mutex> lk(sh->mu);
                sh->cv.wait(lk, [&] { return sh->abort || sh->landed_recorded > prev; });
                if (sh->abort) break;
                lk.unlock();
                if (hipEventSynchronize((*landed)[prev]) != hipSuccess) {
                    set_error(OC_EHIP, "hipEventSynchronize on a landed event failed");
                    break;
                }
            }
            if (aborted()) break;
            const oc_request &r = reqs[it.req];
            const int64_t N = it.chunks ? it.j1 - it.j0 : r.prefix_tokens / c->pool.layout.chunk_tokens;
            const int64_t unit = it.chunks ? (int64_t)L * S : S;
            {
                std::lock_guard<std::mutex> g(wmu);
                chunks_per_piece = std::max<int64_t>(1, c->opts.piece_bytes / unit);
                n_pieces = (N + chunks_per_piece - 1) / chunks_per_piece;
                next_piece = 0;
                pieces_done = 0;
                bytes_done = 0;
                piece_done.assign(n_pieces, 0);
                prefix_pieces = 0;
                cum_before = cum;
                cur_item = k;
            }
            wcv.notify_all();
            int64_t delivered;
            {
                std::unique_lock<std::mutex> lk(wmu);
                wcv.wait(lk, [&] { return pieces_done == n_pieces; });
                cur_item = -1;
                delivered = bytes_done;
            }
            cum += (double)N * unit;
            (*produced_ms)[k] = std::chrono::duration<double, std::milli>(Clock::now() - t0).count();
            roctxMarkA(("ready layer " + std::to_string(it.layer) + " req " + std::to_string(it.req)).c_str());
            {
                std::lock_guard<std::mutex> g(sh->mu);
                sh->delivered[k] = delivered;
                sh->ready = k + 1;
            }
            sh->cv.notify_all();
        }
        {
            std::lock_guard<std::mutex> g(wmu);
            stop = true;
        }
        wcv.notify_all();
        for (auto &t : pool) t.join();
    }
};

// ---- per-request rates (allocation policies) --------------------------------
// Each request is paced by its own clock at its allocated rate, from its
// admission (the epoch boundary oc_epoch_schedule gives it) to its last
// byte: a request that finishes early does not pass its rate on to the
// others in flight; later admissions get it.  The dispatcher hands out
// payload pieces by weighted deficit round robin to the copy threads, which
// copy each piece once its release time has come.  A request's credit grows
// with elapsed time at its rate (the weight), not by a fixed amount per
// round: rounds are uneven in length, and a per-round quantum would hold a
// slow request below its rate whenever its share of a round is smaller than
// the round's length times its rate.  A request starts its next layer only
// when a staging slot is free; its layers are reported to the driver in
// layer order, and the driver lands whichever layer is reported first, so a
// slow request does not hold up a fast one.
struct RateProducer {
    Context *c;
    RunShared *sh;
    const oc_request *reqs;
    int32_t n_reqs, L;
    int64_t S;
    Clock::time_point t0;
    std::vector<double> rate;                // bytes/s per request
    std::vector<double> admit;               // seconds after t0 at which each request's pacing starts
    std::vector<double> *produced_ms;        // per item k = layer * n_reqs + request
    std::vector<hipEvent_t> *landed;         // per item

    struct Piece {
        double release_s;
        int64_t item, j0, j1;
        int slot;
    };
    struct Later {
        bool operator()(const Piece &a, const Piece &b) const { return a.release_s > b.release_s; }
    };
    // lock order: wmu may be held while taking sh->mu, never the reverse
    std::mutex wmu;
    std::condition_variable wcv;
    std::priority_queue<Piece, std::vector<Piece>, Later> heap;
    bool stop = false;
    std::vector<int64_t> pieces_left;        // per item
    std::vector<int64_t> bytes_of;           // per item: bytes its pieces copied
    std::vector<char> complete;              // per item
    std::vector<int32_t> next_report;        // per request: the layer to report next
    std::vector<int> slot_of;                // per item; written before the item is reported

    struct FreeSlot {
        int slot;
        int64_t after_item;                  // its DMA must have landed before reuse (-1: none)
    };
    std::deque<FreeSlot> free_slots;         // guarded by sh->mu

    double now_s() const { return std::chrono::duration<double>(Clock::now() - t0).count(); }
    int64_t item_of(int32_t layer, int32_t r) const { return (int64_t)layer * n_reqs + r; }

    bool aborted() {
        std::lock_guard<std::mutex> g(sh->mu);
        return sh->abort;
    }
    void set_error(int st, const char *msg) {
        std::lock_guard<std::mutex> g(sh->mu);
        if (sh->producer_status == OC_OK) {
            sh->producer_status = st;
            sh->producer_msg = msg;
        }
        sh->cv.notify_all();
    }

    // called with wmu held: hand every finished layer of request r, in layer order, to the driver
    void report_ready(int32_t r) {
        std::lock_guard<std::mutex> g(sh->mu);
        while (next_report[r] < L && complete[item_of(next_report[r], r)]) {
            const int64_t k = item_of(next_report[r], r);
            (*produced_ms)[k] = std::chrono::duration<double, std::milli>(Clock::now() - t0).count();
            roctxMarkA(("ready layer " + std::to_string(next_report[r]) + " req " + std::to_string(r)).c_str());
            sh->delivered[k] = bytes_of[k];
            sh->reported.push_back(k);
            ++next_report[r];
        }
        sh->cv.notify_all();
    }

    // a free slot whose previous DMA has landed, or -1
    int acquire_slot() {
        std::lock_guard<std::mutex> g(sh->mu);
        for (auto it = free_slots.begin(); it != free_slots.end(); ++it) {
            if (it->after_item >= 0 && hipEventQuery((*landed)[it->after_item]) != hipSuccess) continue;
            const int s = it->slot;
            free_slots.erase(it);
            return s;
        }
        return -1;
    }

    void worker() {
        for (;;) {
            Piece pc;
            {
                std::unique_lock<std::mutex> lk(wmu);
                for (;;) {
                    if (stop) return;
                    if (!heap.empty()) {
                        const double wait = heap.top().release_s - now_s();
                        if (wait <= 0.0) {
                            pc = heap.top();
                            heap.pop();
                            break;
                        }
                        wcv.wait_for(lk, std::chrono::duration<double>(std::min(wait, 0.001)));
                    } else {
                        wcv.wait(lk);
                    }
                }
            }
            const int32_t layer = (int32_t)(pc.item / n_reqs), r = (int32_t)(pc.item % n_reqs);
            const int64_t N = reqs[r].prefix_tokens / c->pool.layout.chunk_tokens;
            unsigned char *dst = static_cast<unsigned char *>(c->slots[pc.slot].pinned);
            int64_t copied = 0;
            for (int64_t j = pc.j0; j < pc.j1; ++j) {
                const unsigned char *obj = static_cast<const unsigned char *>(reqs[r].chunk_objects[j]);
                const int64_t len = copy_len(c->opts, layer, j, N, S);
                std::memcpy(dst + j * S, obj + (int64_t)layer * S, (size_t)len);
                copied += len;
            }
            std::lock_guard<std::mutex> g(wmu);
            bytes_of[pc.item] += copied;
            if (--pieces_left[pc.item] == 0) {
                complete[pc.item] = 1;
                report_ready(r);
            }
            wcv.notify_all();
        }
    }

    void run() {
        const int64_t n_items = (int64_t)n_reqs * L;
        const int64_t cpp = std::max<int64_t>(1, c->opts.piece_bytes / S);     // chunks per piece
        pieces_left.assign(n_items, 0);
        bytes_of.assign(n_items, 0);
        complete.assign(n_items, 0);
        next_report.assign(n_reqs, 0);
        slot_of.assign(n_items, -1);
        {
            std::lock_guard<std::mutex> g(sh->mu);
            for (int s = 0; s < (int)c->slots.size(); ++s) free_slots.push_back({s, -1});
        }
        std::vector<int64_t> N(n_reqs), npieces(n_reqs), piece(n_reqs, 0);
        std::vector<int32_t> layer(n_reqs, 0);
        const double lookahead_s = 0.004;   // hand out pieces due within this window
        // credit cap: two pieces beyond what the look-ahead window releases
        std::vector<double> cum(n_reqs, 0.0), deficit(n_reqs, 0.0), credit_cap(n_reqs, 0.0);
        {
            std::lock_guard<std::mutex> g(wmu);
            for (int32_t r = 0; r < n_reqs; ++r) {
                N[r] = reqs[r].prefix_tokens / c->pool.layout.chunk_tokens;
                npieces[r] = (N[r] + cpp - 1) / cpp;
                credit_cap[r] = 2.0 * (double)(cpp * S) + rate[r] * lookahead_s;
                deficit[r] = credit_cap[r];
                for (int32_t l = 0; l < L; ++l) pieces_left[item_of(l, r)] = npieces[r];
                if (N[r] == 0) {            // nothing to deliver: every layer is ready now
                    for (int32_t l = 0; l < L; ++l) complete[item_of(l, r)] = 1;
                    layer[r] = L;
                    report_ready(r);
                }
            }
        }
        std::vector<std::thread> pool;
        if (start_threads(pool, c->opts.producer_threads, [this] { worker(); }) == 0) {
            set_error(OC_ENOMEM, "could not start the producer's copy threads");
            return;
        }
        bool failed = false;
        double last_round = now_s();
        for (;;) {
            const double round_start = now_s(), dt = round_start - last_round;
            last_round = round_start;
            if (aborted()) {
                failed = true;
                break;
            }
            bool all_done = true, progress = false;
            for (int32_t r = 0; r < n_reqs; ++r) {
                if (layer[r] >= L) continue;
                all_done = false;
                if (stops_at(c->opts, layer[r]) && piece[r] == 0) {
                    if (c->opts.fault == OC_FAULT_ABORT) {
                        set_error(OC_EABORT, "producer aborted (injected fault)");
                    } else {      // injected stall: deliver nothing more until the driver gives up
                        std::unique_lock<std::mutex> lk(sh->mu);
                        sh->cv.wait(lk, [&] { return sh->abort; });
                    }
                    failed = true;
                    break;
                }
                deficit[r] = std::min(deficit[r] + rate[r] * dt, credit_cap[r]);
                while (layer[r] < L) {
                    const int64_t j0 = piece[r] * cpp, j1 = std::min(N[r], j0 + cpp);
                    const double bytes = (double)(j1 - j0) * S;
                    if (deficit[r] < bytes) break;
                    const double release = admit[r] + (cum[r] + bytes) / rate[r];
                    if (release > now_s() + lookahead_s) break;
                    const int64_t k = item_of(layer[r], r);
                    if (piece[r] == 0) {
                        const int s = acquire_slot();
                        if (s < 0) break;
                        slot_of[k] = s;
                    }
                    {
                        std::lock_guard<std::mutex> g(wmu);
                        heap.push({release, k, j0, j1, slot_of[k]});
                    }
                    wcv.notify_all();
                    cum[r] += bytes;
                    deficit[r] -= bytes;
                    progress = true;
                    if (++piece[r] == npieces[r]) {
                        ++layer[r];
                        piece[r] = 0;
                    }
                }
            }
            if (failed || all_done) break;
            if (!progress) {     // wait for a slot to come back or the next release window
                std::unique_lock<std::mutex> lk(sh->mu);
                sh->cv.wait_for(lk, std::chrono::microseconds(250));
            }
        }
        // let the copies already handed out finish, unless the run is stopped
        if (!failed) {
            for (;;) {
                std::unique_lock<std::mutex> lk(wmu);
                const bool finished = wcv.wait_for(lk, std::chrono::milliseconds(1), [&] {
                    if (!heap.empty()) return false;
                    for (int64_t k = 0; k < n_items; ++k)
                        if (pieces_left[k] > 0) return false;
                    return true;
                });
                lk.unlock();
                if (finished || aborted()) break;
            }
        }
        {
            std::lock_guard<std::mutex> g(wmu);
            stop = true;
        }
        wcv.notify_all();
        for (auto &t : pool) t.join();
    }
};

static int validate_requests(Context *c, const oc_request *reqs, int32_t n) {
    const oc_layout &l = c->pool.layout;
    const int mode = c->opts.mode;
    for (int32_t i = 0; i < n; ++i) {
        const oc_request &r = reqs[i];
        const std::string who = "request " + std::to_string(i) + ": ";
        if (!r.block_table) return fail(OC_EINVAL, who + "block_table is NULL");
        if (r.prefix_tokens < 0 || r.suffix_tokens < 1) return fail(OC_EINVAL, who + "bad lengths");
        if (r.prefix_tokens != r.block_table->num_tokens)
            return fail(OC_ESHAPE, who + "prefix_tokens differs from the block table's num_tokens");
        if (r.prefix_tokens % l.chunk_tokens) return fail(OC_ESHAPE, who + "prefix is not a whole number of chunks");
        if (r.prefix_tokens > c->max_prefix || r.suffix_tokens > c->max_suffix)
            return fail(OC_ERANGE, who + "longer than the context was created for");
        if (!(r.arrival_s >= 0.0) || !std::isfinite(r.arrival_s))
            return fail(OC_EINVAL, who + "arrival_s must be >= 0 and finite");
        if (r.arrival_s > 0.0 && !(mode == OC_MODE_PRODUCER && c->opts.alloc_policy != OC_ALLOC_FIFO))
            return fail(OC_EINVAL, who + "arrival_s > 0 needs the producer mode with an allocation policy");
        const int64_t need = (r.prefix_tokens + l.page_size - 1) / l.page_size;
        if (r.block_table->num_entries < need) return fail(OC_ERANGE, who + "block table too short");
        if (need > 0 && !r.block_table->pages) return fail(OC_EINVAL, who + "NULL block table pages");
        if (c->opts.append_suffix && check_append_table(r.block_table, l, r.suffix_tokens) != OC_OK)
            return fail(OC_ERANGE, who + oc_last_error());
        if (!r.q || !r.k_new || !r.v_new || !r.out) return fail(OC_EINVAL, who + "NULL q/k_new/v_new/out");
        if (!aligned(r.q, 16) || !aligned(r.k_new, 16) || !aligned(r.v_new, 16) || !aligned(r.out, 16))
            return fail(OC_EALIGN, who + "q/k_new/v_new/out must be 16-byte aligned");
        if (mode == OC_MODE_DEVICE_STAGED && r.prefix_tokens > 0) {
            if (!r.device_payload) return fail(OC_EINVAL, who + "DEVICE_STAGED needs device_payload");
            if (!aligned(r.device_payload, 16)) return fail(OC_EALIGN, who + "device_payload must be 16-byte aligned");
        }
        if (mode == OC_MODE_PRODUCER && r.prefix_tokens > 0) {
            if (!r.chunk_objects) return fail(OC_EINVAL, who + "PRODUCER needs chunk_objects");
            const int64_t N = r.prefix_tokens / l.chunk_tokens;
            for (int64_t j = 0; j < N; ++j)
                if (!r.chunk_objects[j]) return fail(OC_EINVAL, who + "NULL chunk object");
        }
    }
    return OC_OK;
}

static double ev_ms(hipEvent_t a, hipEvent_t b) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return -1.0;
    return ms;
}

static int run_pipeline(Context *c, const oc_request *reqs, int32_t n_reqs, oc_request_stats *stats) {
    const DeviceScope on_device(c->device);
    const TraceRange trace_run("oc_pipeline_run");
    const oc_layout &l = c->pool.layout;
    const int32_t L = l.num_layers;
    const int mode = c->opts.mode;
    const int64_t b_tok = 2LL * l.num_kv_heads * l.head_dim * 2;     // bytes per token per layer
    const int64_t S = b_tok * l.chunk_tokens;

    // Each request computes on the compute stream, or with emulated windows on
    // a stream of its own; every stream in use gets its own attention
    // workspace and rest-of-layer buffers, since their work may overlap.
    const bool emu = c->opts.emulate_compute != 0;
    const int64_t n_streams = emu ? n_reqs : 1;
    // When every request is delivered layer-major on one schedule and computes
    // on the compute stream, each layer's attention is one launch over all
    // of them (decided below, once the deliveries are known); its plans split
    // keys for all their row tiles together.
    std::vector<AttnPlan> bplan(n_reqs);
    std::vector<size_t> bws_off(n_reqs, 0);
    size_t ws_need = 0, bws_need = 0;
    int64_t max_ts = 0;
    for (int32_t i = 0; i < n_reqs; ++i) {
        AttnPlan p;
        plan_attention(l, reqs[i].prefix_tokens, reqs[i].suffix_tokens, &p);
        ws_need = std::max(ws_need, p.total);
        max_ts = std::max(max_ts, reqs[i].suffix_tokens);
    }
    if (n_reqs >= 2 && n_reqs <= MAX_ATTN_BATCH) {
        std::vector<int64_t> tp(n_reqs), ts(n_reqs);
        for (int32_t i = 0; i < n_reqs; ++i) {
            tp[i] = reqs[i].prefix_tokens;
            ts[i] = reqs[i].suffix_tokens;
        }
        plan_attention_batch(l, tp.data(), ts.data(), n_reqs, bplan.data());
        for (int32_t i = 0; i < n_reqs; ++i) {
            bws_off[i] = bws_need;
            bws_need += (bplan[i].total + 255) / 256 * 256;
        }
        ws_need = std::max(ws_need, bws_need);
    }
    const size_t ws_stride = (ws_need + 255) / 256 * 256;
    if (ws_stride * n_streams > c->ws_bytes) {
        if (c->ws) OC_HIP(hipFree(c->ws));
        c->ws = nullptr;
        c->ws_bytes = 0;
        if (hipMalloc(&c->ws, ws_stride * n_streams) != hipSuccess)
            return fail(OC_ENOMEM, "attention workspace allocation failed");
        c->ws_bytes = ws_stride * n_streams;
    }
    size_t loff[5] = {0, 0, 0, 0, 0};
    const size_t lb_stride = c->has_layer ? layer_buffer_bytes(l, c->lw.ffn_dim, max_ts, loff) : 0;
    if (lb_stride * n_streams > c->lbuf_bytes) {
        if (c->lbuf) OC_HIP(hipFree(c->lbuf));
        c->lbuf = nullptr;
        c->lbuf_bytes = 0;
        if (hipMalloc(&c->lbuf, lb_stride * n_streams) != hipSuccess)
            return fail(OC_ENOMEM, "rest-of-layer buffer allocation failed");
        c->lbuf_bytes = lb_stride * n_streams;
    }

    // delivery of each request (eq. (2)); only the producer has an order to choose
    std::vector<int32_t> deliv(n_reqs, OC_DELIVERY_LAYERWISE);
    const int64_t obj_bytes = (int64_t)L * S;     // one whole chunk object
    int n_cw = 0;
    if (mode == OC_MODE_PRODUCER)
        for (int32_t r = 0; r < n_reqs; ++r) {
            const int64_t N = reqs[r].prefix_tokens / l.chunk_tokens;
            const double W = (double)N * (double)obj_bytes;
            if (N > 0 && (c->opts.delivery == OC_DELIVERY_CHUNKWISE ||
                          (c->opts.delivery == OC_DELIVERY_AUTO && W < c->opts.theta_bytes))) {
                deliv[r] = OC_DELIVERY_CHUNKWISE;
                ++n_cw;
            }
        }
    if (emu)
        for (int32_t r = 0; r < n_reqs; ++r)
            if (!(reqs[r].layer_compute_s >= 0.0) || reqs[r].layer_compute_s > OC_MAX_WINDOW_S)
                return fail(OC_EINVAL, "emulated compute window must be in [0, 10] seconds");
    // the stream each request's attention (and emulated window) runs on
    while (emu && (int32_t)c->req_streams.size() < n_reqs) {
        hipStream_t st;
        OC_HIP(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));   // default priority
        c->req_streams.push_back(st);
    }
    auto stream_of = [&](int32_t r) { return emu ? c->req_streams[r] : c->compute; };
    if (n_cw > 0 && c->opts.alloc_policy != OC_ALLOC_FIFO)
        return fail(OC_EINVAL, "a request falls on the chunkwise side of theta_bytes, and allocation policies "
                               "schedule layerwise requests only (use OC_ALLOC_FIFO)");
    if (n_cw > 0 && (int64_t)c->slot_bytes < obj_bytes)
        return fail(OC_EINVAL, "staging slots hold less than one chunk object: create the context with a "
                               "chunkwise-capable delivery");

    // items: every chunkwise request's object groups (as many whole objects as
    // a slot holds), then the layerwise requests layer-major, request-minor
    std::vector<Item> items;
    std::vector<int64_t> last_group(n_reqs, -1), item_of((size_t)n_reqs * L, -1);
    const int64_t per_group = n_cw > 0 ? (int64_t)c->slot_bytes / obj_bytes : 1;
    for (int32_t r = 0; r < n_reqs; ++r) {
        if (deliv[r] != OC_DELIVERY_CHUNKWISE) continue;
        const int64_t N = reqs[r].prefix_tokens / l.chunk_tokens;
        for (int64_t j0 = 0; j0 < N; j0 += per_group) {
            items.push_back({0, r, true, j0, std::min(N, j0 + per_group)});
            last_group[r] = (int64_t)items.size() - 1;
        }
    }
    for (int32_t layer = 0; layer < L; ++layer)
        for (int32_t r = 0; r < n_reqs; ++r)
            if (deliv[r] == OC_DELIVERY_LAYERWISE) {
                item_of[(size_t)r * L + layer] = (int64_t)items.size();
                items.push_back({layer, r});
            }
    const int64_t n_items = (int64_t)items.size();

    // events: start, landed/ingested per item, done per (request, layer)
    const size_t n_done = (size_t)n_reqs * L;
    const size_t n_ev = 1 + 2 * (size_t)n_items + n_done;
    while (c->events.size() < n_ev) {
        hipEvent_t e;
        OC_HIP(hipEventCreate(&e));
        c->events.push_back(e);
    }
    hipEvent_t ev_start = c->events[0];
    std::vector<hipEvent_t> landed(c->events.begin() + 1, c->events.begin() + 1 + n_items);
    std::vector<hipEvent_t> ingested(c->events.begin() + 1 + n_items, c->events.begin() + 1 + 2 * n_items);
    std::vector<hipEvent_t> done(c->events.begin() + 1 + 2 * n_items, c->events.begin() + 1 + 2 * n_items + n_done);
    std::vector<double> produced(n_items, -1.0);

    // one layer's compute for request `ri` on `st`: attention, then the suffix
    // append and the rest of the layer when asked for
    std::string layer_msg;       // why the rest of the layer failed to enqueue
    auto attn_args = [&](int32_t ri, int32_t layer, unsigned char *ws) {
        const oc_request &r = reqs[ri];
        AttnArgs a{};
        const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
        const uint16_t *base = static_cast<const uint16_t *>(c->pool.base);
        const int64_t q_stride = r.suffix_tokens * l.num_q_heads * l.head_dim;
        const int64_t kv_stride = r.suffix_tokens * l.num_kv_heads * l.head_dim;
        a.q = static_cast<const uint16_t *>(r.q) + layer * q_stride;
        a.k_new = static_cast<const uint16_t *>(r.k_new) + layer * kv_stride;
        a.v_new = static_cast<const uint16_t *>(r.v_new) + layer * kv_stride;
        a.out = static_cast<uint16_t *>(r.out) + layer * q_stride;
        a.pool_k = base + ((int64_t)layer * 2 + 0) * l.num_pages * block;
        a.pool_v = base + ((int64_t)layer * 2 + 1) * l.num_pages * block;
        a.pages = r.block_table->pages;
        a.ws = ws;
        return a;
    };
    // after a request's attention: the suffix append and the rest of the layer
    auto after_attention = [&](int32_t ri, int32_t layer, const AttnArgs &a, hipStream_t st) -> hipError_t {
        const oc_request &r = reqs[ri];
        hipError_t e = hipSuccess;
        if (c->opts.append_suffix)
            e = launch_append(append_args(&c->pool, r.block_table, layer, a.k_new, a.v_new, r.suffix_tokens), st);
        if (e == hipSuccess && c->has_layer) {
            unsigned char *lb = static_cast<unsigned char *>(c->lbuf) + (emu ? ri : 0) * lb_stride;
            const oc_layer_buffers bufs{lb + loff[0], lb + loff[1], lb + loff[2], lb + loff[3], lb + loff[4]};
            if (launch_rest_of_layer(layer_args(l, c->lw, layer, a.out, r.suffix_tokens, bufs), st) != OC_OK) {
                layer_msg = oc_last_error();
                return hipErrorLaunchFailure;
            }
        }
        return e;
    };
    // one layer's compute for request `ri` on `st`
    auto enqueue_attention = [&](int32_t ri, int32_t layer, hipStream_t st) -> hipError_t {
        const oc_request &r = reqs[ri];
        AttnPlan p;
        plan_attention(l, r.prefix_tokens, r.suffix_tokens, &p);
        const AttnArgs a = attn_args(ri, layer, static_cast<unsigned char *>(c->ws) + (emu ? ri : 0) * ws_stride);
        hipError_t e = launch_attention(p, a, st);
        return e == hipSuccess ? after_attention(ri, layer, a, st) : e;
    };
    // one layer's compute for every request: one attention launch over all
    auto enqueue_layer_batch = [&](int32_t layer, hipStream_t st) -> hipError_t {
        std::vector<AttnArgs> args(n_reqs);
        for (int32_t ri = 0; ri < n_reqs; ++ri)
            args[ri] = attn_args(ri, layer, static_cast<unsigned char *>(c->ws) + bws_off[ri]);
        hipError_t e = launch_attention_batch(bplan.data(), args.data(), n_reqs, st);
        for (int32_t ri = 0; ri < n_reqs && e == hipSuccess; ++ri) e = after_attention(ri, layer, args[ri], st);
        return e;
    };

    OC_HIP(hipStreamSynchronize(c->copy));
    OC_HIP(hipStreamSynchronize(c->compute));
    // The context's streams are non-blocking, so nothing orders them after
    // what the caller enqueued on the null stream (filling the pool, copying
    // tables and suffix tensors): wait for that work on the device first.
    OC_HIP(hipEventRecord(c->caller_done, nullptr));
    OC_HIP(hipStreamWaitEvent(c->copy, c->caller_done, 0));
    OC_HIP(hipStreamWaitEvent(c->compute, c->caller_done, 0));
    if (emu)
        for (int32_t r = 0; r < n_reqs; ++r) OC_HIP(hipStreamWaitEvent(c->req_streams[r], c->caller_done, 0));

    // per-request rates under the shared budget (allocation policies)
    const bool by_rate = mode == OC_MODE_PRODUCER && c->opts.alloc_policy != OC_ALLOC_FIFO;
    int64_t batch_grid = 0;   // workgroups of one batched launch
    if (n_reqs >= 2 && n_reqs <= MAX_ATTN_BATCH)
        for (int32_t i = 0; i < n_reqs; ++i) batch_grid += attention_grid(bplan[i]);
    const bool batched = !c->opts.attention_per_request && !emu && !by_rate && n_cw == 0 && n_reqs >= 2 &&
                         n_reqs <= MAX_ATTN_BATCH && batch_grid <= attention_max_grid();
    std::vector<double> req_rate(n_reqs, 0.0), req_admit(n_reqs, 0.0);
    if (by_rate) {
        // rates and admissions by scheduling epoch; with every arrival at
        // the start this is one epoch, oc_bandwidth_allocate over all of them
        std::vector<double> s_i, c_i, a_i;
        std::vector<int32_t> who;
        for (int32_t r = 0; r < n_reqs; ++r) {
            req_admit[r] = reqs[r].arrival_s;      // nothing to deliver: admitted on arrival
            if (reqs[r].prefix_tokens > 0) {
                who.push_back(r);
                s_i.push_back((double)reqs[r].prefix_tokens * (double)b_tok);
                c_i.push_back(reqs[r].layer_compute_s);
                a_i.push_back(reqs[r].arrival_s);
            }
        }
        if (!who.empty()) {
            std::vector<double> out(who.size()), adm(who.size());
            const int rc = oc_epoch_schedule(c->opts.alloc_policy, (int32_t)who.size(), s_i.data(), c_i.data(), L,
                                             a_i.data(), c->opts.rate_bytes_per_s, c->opts.margin_bytes_per_s,
                                             c->opts.epoch_s, out.data(), adm.data());
            if (rc) return rc;
            for (size_t i = 0; i < who.size(); ++i) {
                req_rate[who[i]] = out[i];
                req_admit[who[i]] = adm[i];
            }
        }
    }

    RunShared sh;
    sh.delivered.assign(n_items, 0);
    Producer prod{};
    RateProducer rprod{};
    std::thread producer_thread;
    // however the run ends (an exception included), the producer is stopped
    // and joined before the state it uses goes away
    struct StopOnExit {
        std::thread &t;
        RunShared &sh;
        ~StopOnExit() {
            if (!t.joinable()) return;
            {
                std::lock_guard<std::mutex> g(sh.mu);
                sh.abort = true;
            }
            sh.cv.notify_all();
            t.join();
        }
    } stop_on_exit{producer_thread, sh};
    const hipStream_t first = mode == OC_MODE_HBM_RESIDENT ? c->compute : c->copy;
    OC_HIP(hipEventRecord(ev_start, first));
    if (mode != OC_MODE_HBM_RESIDENT) OC_HIP(hipStreamWaitEvent(c->compute, ev_start, 0));
    if (emu)
        for (int32_t r = 0; r < n_reqs; ++r) OC_HIP(hipStreamWaitEvent(c->req_streams[r], ev_start, 0));
    const Clock::time_point t0 = Clock::now();

    if (by_rate) {
        rprod.c = c;
        rprod.sh = &sh;
        rprod.reqs = reqs;
        rprod.n_reqs = n_reqs;
        rprod.L = L;
        rprod.S = S;
        rprod.t0 = t0;
        rprod.rate = req_rate;
        rprod.admit = req_admit;
        rprod.produced_ms = &produced;
        rprod.landed = &landed;
        producer_thread = std::thread([&rprod] { rprod.run(); });
    } else if (mode == OC_MODE_PRODUCER) {
        prod.c = c;
        prod.sh = &sh;
        prod.reqs = reqs;
        prod.items = &items;
        prod.t0 = t0;
        prod.produced_ms = &produced;
        prod.landed = &landed;
        prod.rate = c->opts.rate_bytes_per_s;
        prod.S = S;
        prod.L = L;
        producer_thread = std::thread([&prod] { prod.run(); });
    }

    int status = OC_OK;
    std::string msg;
    // a payload shorter than its item is never ingested: the run stops there
    auto short_payload = [&](const Item &it, int64_t got, int64_t want) {
        const std::string what = it.chunks ? "chunks " + std::to_string(it.j0) + ".." + std::to_string(it.j1 - 1)
                                           : "layer " + std::to_string(it.layer);
        status = OC_ESHORT;
        msg = what + " of request " + std::to_string(it.req) + ": the producer delivered " + std::to_string(got) +
              " of " + std::to_string(want) + " bytes";
    };
    for (int64_t step = 0; step < n_items && status == OC_OK; ++step) {
        int64_t k = step;
        int64_t got = 0;   // bytes the producer reports for item k
        if (by_rate) {     // the next layer any request has ready, in the order they became ready
            std::unique_lock<std::mutex> lk(sh.mu);
            const auto deadline = Clock::now() + std::chrono::milliseconds(c->opts.timeout_ms);
            const bool ok = sh.cv.wait_until(lk, deadline, [&] { return !sh.reported.empty() || sh.producer_status != OC_OK; });
            if (sh.producer_status != OC_OK) {
                status = sh.producer_status;
                msg = sh.producer_msg;
                break;
            }
            if (!ok) {
                status = OC_ETIMEOUT;
                msg = "no layer arrived within " + std::to_string(c->opts.timeout_ms) + " ms";
                break;
            }
            k = sh.reported.front();
            sh.reported.pop_front();
            got = sh.delivered[k];
        }
        const Item it = items[k];
        const TraceRange trace_item(it.chunks ? "chunks " + std::to_string(it.j0) + ".." + std::to_string(it.j1 - 1) +
                                                    " req " + std::to_string(it.req)
                                              : "layer " + std::to_string(it.layer) + " req " + std::to_string(it.req));
        const oc_request &r = reqs[it.req];
        const int64_t layer_bytes = r.prefix_tokens * b_tok;
        const int64_t N = r.prefix_tokens / l.chunk_tokens;
        const void *payload = nullptr;
        if (it.chunks) {
            // a group of whole chunk objects: land it, ingest every layer of
            // it; after the request's last group, all its layers compute
            {
                std::unique_lock<std::mutex> lk(sh.mu);
                const auto deadline = Clock::now() + std::chrono::milliseconds(c->opts.timeout_ms);
                const bool ok = sh.cv.wait_until(lk, deadline, [&] { return sh.ready > k || sh.producer_status != OC_OK; });
                if (sh.producer_status != OC_OK) {
                    status = sh.producer_status;
                    msg = sh.producer_msg;
                    break;
                }
                if (!ok) {
                    status = OC_ETIMEOUT;
                    msg = "chunks " + std::to_string(it.j0) + ".." + std::to_string(it.j1 - 1) + " of request " +
                          std::to_string(it.req) + " did not arrive within " + std::to_string(c->opts.timeout_ms) +
                          " ms";
                    break;
                }
                got = sh.delivered[k];
            }
            if (got != (it.j1 - it.j0) * obj_bytes) {
                short_payload(it, got, (it.j1 - it.j0) * obj_bytes);
                break;
            }
            Slot &s = c->slots[k % c->slots.size()];
            hipError_t e = hipMemcpyAsync(s.device, s.pinned, (size_t)((it.j1 - it.j0) * obj_bytes),
                                          hipMemcpyHostToDevice, c->copy);
            if (e == hipSuccess) e = hipEventRecord(landed[k], c->copy);
            {
                std::lock_guard<std::mutex> g(sh.mu);
                sh.landed_recorded = k + 1;
            }
            sh.cv.notify_all();
            if (e == hipSuccess)
                e = launch_chunks_ingest(chunks_ingest_args(&c->pool, r.block_table, s.device, it.j0, it.j1 - it.j0),
                                         c->copy);
            if (e == hipSuccess) e = hipEventRecord(ingested[k], c->copy);
            if (e == hipSuccess && k == last_group[it.req]) {
                const hipStream_t cs = stream_of(it.req);
                e = hipStreamWaitEvent(cs, ingested[k], 0);
                for (int32_t layer = 0; layer < L && e == hipSuccess; ++layer) {
                    e = enqueue_attention(it.req, layer, cs);
                    if (e == hipSuccess && emu) e = launch_compute_window(r.layer_compute_s, cs);
                    if (e == hipSuccess) e = hipEventRecord(done[(size_t)it.req * L + layer], cs);
                }
            }
            if (e != hipSuccess) {
                status = layer_msg.empty() ? hip_fail(e, "enqueueing a chunk group") : fail(OC_EHIP, layer_msg);
                msg = oc_last_error();
                break;
            }
            continue;
        }
        if (by_rate) {
            if (got != layer_bytes) {
                short_payload(it, got, layer_bytes);
                break;
            }
            if (layer_bytes > 0) {
                const int slot = rprod.slot_of[k];
                Slot &s = c->slots[slot];
                hipError_t e = hipMemcpyAsync(s.device, s.pinned, (size_t)layer_bytes, hipMemcpyHostToDevice, c->copy);
                if (e == hipSuccess) e = hipEventRecord(landed[k], c->copy);
                {
                    std::lock_guard<std::mutex> g(sh.mu);
                    rprod.free_slots.push_back({slot, k});   // reusable once this DMA has landed
                }
                sh.cv.notify_all();
                if (e != hipSuccess) {
                    status = hip_fail(e, "landing a layer payload");
                    msg = oc_last_error();
                    break;
                }
                payload = s.device;
            } else {
                hipError_t e = hipEventRecord(landed[k], c->copy);
                if (e != hipSuccess) {
                    status = hip_fail(e, "hipEventRecord");
                    msg = oc_last_error();
                    break;
                }
            }
        } else if (mode == OC_MODE_PRODUCER) {
            // land the payload in spans as the producer completes its leading
            // bytes, so the copy of a layer overlaps its production; the
            // ingest still waits for the whole layer
            Slot &s = c->slots[k % c->slots.size()];
            const int64_t span = landing_span(c->opts, layer_bytes);
            const unsigned char *src = static_cast<const unsigned char *>(s.pinned);
            unsigned char *dst = static_cast<unsigned char *>(s.device);
            const auto deadline = Clock::now() + std::chrono::milliseconds(c->opts.timeout_ms);
            int64_t sent = 0;
            bool whole = false;
            hipError_t e = hipSuccess;
            while (!whole && e == hipSuccess) {
                int64_t avail;
                {
                    std::unique_lock<std::mutex> lk(sh.mu);
                    const bool ok = sh.cv.wait_until(lk, deadline, [&] {
                        return sh.ready > k ||
                               (sh.part_item == k && sh.part_bytes >= std::min(layer_bytes, (sent / span + 1) * span)) ||
                               sh.producer_status != OC_OK;
                    });
                    if (sh.producer_status != OC_OK) {
                        status = sh.producer_status;
                        msg = sh.producer_msg;
                        break;
                    }
                    if (!ok) {
                        status = OC_ETIMEOUT;
                        msg = "layer " + std::to_string(it.layer) + " of request " + std::to_string(it.req) +
                              " did not arrive within " + std::to_string(c->opts.timeout_ms) + " ms";
                        break;
                    }
                    whole = sh.ready > k;
                    got = sh.delivered[k];
                    avail = whole ? layer_bytes : sh.part_bytes;
                }
                if (whole && got != layer_bytes) {
                    short_payload(it, got, layer_bytes);     // landed in part, never ingested
                    break;
                }
                if (avail > sent) {
                    e = hipMemcpyAsync(dst + sent, src + sent, (size_t)(avail - sent), hipMemcpyHostToDevice, c->copy);
                    sent = avail;
                }
            }
            if (status != OC_OK) break;
            if (e == hipSuccess) e = hipEventRecord(landed[k], c->copy);
            {
                std::lock_guard<std::mutex> g(sh.mu);
                sh.landed_recorded = k + 1;
            }
            sh.cv.notify_all();
            if (e != hipSuccess) {
                status = hip_fail(e, "landing a layer payload");
                msg = oc_last_error();
                break;
            }
            payload = s.device;
        } else if (mode == OC_MODE_DEVICE_STAGED) {
            payload = static_cast<const unsigned char *>(r.device_payload) + (int64_t)it.layer * layer_bytes;
            hipError_t e = hipEventRecord(landed[k], c->copy);
            if (e != hipSuccess) {
                status = hip_fail(e, "hipEventRecord");
                msg = oc_last_error();
                break;
            }
        }
        hipError_t e = hipSuccess;
        hipStream_t attn_stream = stream_of(it.req);
        if (mode != OC_MODE_HBM_RESIDENT) {
            if (N > 0) {
                oc_kv_pool pool = c->pool;
                oc_block_table bt = *r.block_table;
                IngestArgs a{};
                const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
                uint16_t *base = static_cast<uint16_t *>(pool.base);
                a.staging = static_cast<const uint16_t *>(payload);
                a.pool_k = base + ((int64_t)it.layer * 2 + 0) * l.num_pages * block;
                a.pool_v = base + ((int64_t)it.layer * 2 + 1) * l.num_pages * block;
                a.pages = bt.pages;
                a.num_tokens = bt.num_tokens;
                a.G = l.chunk_tokens;
                a.n_kv = l.num_kv_heads;
                a.d = l.head_dim;
                a.Ps = l.page_size;
                e = launch_ingest(a, (bt.num_tokens + l.page_size - 1) / l.page_size, c->copy, step > 0);
            }
            if (e == hipSuccess) e = hipEventRecord(ingested[k], c->copy);
            // batched: the copy stream runs in order, so the layer's last
            // ingest covers the others (each wait and event marker costs
            // the stream a few microseconds)
            if (e == hipSuccess && (!batched || it.req == n_reqs - 1))
                e = hipStreamWaitEvent(attn_stream, ingested[k], 0);
        } else if (!batched || it.req == 0) {    // batched: one pair of markers per layer
            e = hipEventRecord(landed[k], attn_stream);
            if (e == hipSuccess) e = hipEventRecord(ingested[k], attn_stream);
        }
        if (batched) {
            // the layer's last request: one launch for all of them, whose
            // ingests the compute stream has waited for item by item
            if (e == hipSuccess && it.req == n_reqs - 1) {
                e = enqueue_layer_batch(it.layer, attn_stream);
                if (e == hipSuccess) e = hipEventRecord(done[(size_t)(n_reqs - 1) * L + it.layer], attn_stream);
            }
        } else {
            if (e == hipSuccess) e = enqueue_attention(it.req, it.layer, attn_stream);
            if (e == hipSuccess && emu) e = launch_compute_window(r.layer_compute_s, attn_stream);
            if (e == hipSuccess) e = hipEventRecord(done[(size_t)it.req * L + it.layer], attn_stream);
        }
        if (e != hipSuccess) {
            status = layer_msg.empty() ? hip_fail(e, "enqueueing a layer") : fail(OC_EHIP, layer_msg);
            msg = oc_last_error();
            break;
        }
    }

    // stop the producer, then drain whatever was enqueued
    {
        std::lock_guard<std::mutex> g(sh.mu);
        sh.abort = sh.abort || status != OC_OK;
    }
    sh.cv.notify_all();
    if (producer_thread.joinable()) {
        if (status == OC_OK) {
            producer_thread.join();
            if (sh.producer_status != OC_OK) {
                status = sh.producer_status;
                msg = sh.producer_msg;
            }
        } else {
            {
                std::lock_guard<std::mutex> g(sh.mu);
                sh.abort = true;
            }
            sh.cv.notify_all();
            producer_thread.join();
        }
    }
    hipError_t e1 = hipStreamSynchronize(c->copy);
    hipError_t e2 = hipStreamSynchronize(c->compute);
    for (int32_t r = 0; emu && r < n_reqs; ++r) {
        const hipError_t e3 = hipStreamSynchronize(c->req_streams[r]);
        if (e2 == hipSuccess) e2 = e3;
    }
    if (status != OC_OK) return fail(status, msg);
    if (e1 != hipSuccess) return hip_fail(e1, "draining the copy stream");
    if (e2 != hipSuccess) return hip_fail(e2, "draining the compute stream");

    // batched layers share one done event (the last request's) and, with
    // the KV resident, one pair of landed/ingested markers (the first's)
    double last = 0.0;
    for (int32_t r = 0; r < n_reqs; ++r)
        for (int32_t layer = 0; layer < L; ++layer) {
            const double t_done = ev_ms(ev_start, done[(size_t)(batched ? n_reqs - 1 : r) * L + layer]);
            last = std::max(last, t_done);
            if (!stats) continue;
            // a chunkwise request's layers all became usable with its last group
            const int64_t k = deliv[r] == OC_DELIVERY_CHUNKWISE ? last_group[r] : item_of[(size_t)r * L + layer];
            const int64_t k_marker = batched && mode == OC_MODE_HBM_RESIDENT ? item_of[(size_t)layer] : k;
            oc_request_stats &st = stats[r];
            if (layer == L - 1) st.ttft_ms = t_done - reqs[r].arrival_s * 1e3;
            if (st.produced_ms) st.produced_ms[layer] = produced[k];
            if (st.landed_ms) st.landed_ms[layer] = mode == OC_MODE_HBM_RESIDENT ? 0.0 : ev_ms(ev_start, landed[k]);
            if (st.ingested_ms) st.ingested_ms[layer] = ev_ms(ev_start, ingested[k_marker]);
            if (st.done_ms) st.done_ms[layer] = t_done;
            st.rate_bytes_per_s = req_rate[r];
            st.delivery = deliv[r];
            st.admitted_ms = req_admit[r] * 1e3;
        }
    c->last_ms = last;
    return OC_OK;
}

}  // namespace oc

using namespace oc;

extern "C" {

static int context_create_body(int device, const oc_kv_pool *kv_pool, const oc_pipeline_opts *opts,
                               int64_t max_prefix_tokens, int64_t max_suffix_tokens, void **ctx) {
    clear_error();
    if (!kv_pool || !ctx) return fail(OC_EINVAL, "kv_pool and ctx must not be NULL");
    *ctx = nullptr;
    if (max_prefix_tokens < 0 || max_suffix_tokens < 1) return fail(OC_EINVAL, "bad maximum lengths");
    const oc_layout &l = kv_pool->layout;
    // OC_ESHAPE for the layout, OC_ERANGE for lengths past the kernels' limits
    if (int rc = check_attention_args(l, max_prefix_tokens, max_suffix_tokens))
        return fail(rc, std::string("unsupported layout or lengths: ") + oc_last_error());
    if (check_copy_pieces(max_prefix_tokens * 2 * l.num_kv_heads * (l.head_dim / 8), "layer payload"))
        return fail(OC_ERANGE, oc_last_error());
    if (!kv_pool->base || !aligned(kv_pool->base, 16)) return fail(OC_EALIGN, "pool base must be 16-byte aligned");
    // released (streams, events, memory) on every early return
    std::unique_ptr<Context, void (*)(Context *)> hold(new Context(), release);
    Context *c = hold.get();
    c->device = device;
    c->pool = *kv_pool;
    c->opts = opts ? *opts : oc_pipeline_opts{};
    int rc = fill_defaults(c->opts);
    if (rc) return rc;
    if (c->opts.layer_weights) {
        if ((rc = check_layer_weights(l, c->opts.layer_weights))) return rc;
        c->has_layer = true;
        c->lw = *c->opts.layer_weights;
        c->opts.layer_weights = &c->lw;
    }
    c->max_prefix = max_prefix_tokens;
    c->max_suffix = max_suffix_tokens;
    c->slot_bytes = (size_t)max_prefix_tokens * 2 * l.num_kv_heads * l.head_dim * 2;
    if (c->opts.delivery != OC_DELIVERY_LAYERWISE && max_prefix_tokens > 0) {
        // a slot must hold at least one whole chunk object (L*S bytes)
        const size_t obj = (size_t)l.num_layers * 2 * l.chunk_tokens * l.num_kv_heads * l.head_dim * 2;
        c->slot_bytes = std::max(c->slot_bytes, obj);
    }
    // the producer's ring always has its slots, even for requests that bring
    // no cached prefix (the driver and producer index the ring per item)
    if (c->opts.mode == OC_MODE_PRODUCER) c->slot_bytes = std::max<size_t>(c->slot_bytes, 256);
    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || device < 0 || device >= n_dev)
        return fail(OC_EINVAL, "no such device");
    const DeviceScope on_device(device);
    // default-priority, non-blocking streams
    if (hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking) != hipSuccess ||
        hipStreamCreateWithFlags(&c->compute, hipStreamNonBlocking) != hipSuccess)
        return fail(OC_EHIP, "stream creation failed");
    if (hipEventCreateWithFlags(&c->caller_done, hipEventDisableTiming) != hipSuccess)
        return fail(OC_EHIP, "event creation failed");
    if (c->opts.mode == OC_MODE_PRODUCER) {
        c->slots.resize((size_t)c->opts.slots);
        for (auto &s : c->slots) {
            if (hipHostMalloc(&s.pinned, c->slot_bytes, hipHostMallocDefault) != hipSuccess ||
                hipMalloc(&s.device, c->slot_bytes) != hipSuccess)
                return fail(OC_ENOMEM, "staging slot allocation failed");
        }
        // Touch the ring once now, each pinned page by the host and each slot
        // by one DMA: a fresh ring's first pass is otherwise several times
        // slower (the producer's first copies into it, and the first DMAs
        // from it), which would delay the first run's layers by tens of ms.
        for (auto &s : c->slots) {
            prefault(static_cast<unsigned char *>(s.pinned), c->slot_bytes, c->opts.producer_threads);
            if (hipMemcpyAsync(s.device, s.pinned, c->slot_bytes, hipMemcpyHostToDevice, c->copy) != hipSuccess)
                return fail(OC_EHIP, "staging slot warm-up copy failed");
        }
        if (hipStreamSynchronize(c->copy) != hipSuccess) return fail(OC_EHIP, "staging slot warm-up copy failed");
    }
    AttnPlan p;
    plan_attention(l, max_prefix_tokens, max_suffix_tokens, &p);
    if (hipMalloc(&c->ws, p.total) != hipSuccess) return fail(OC_ENOMEM, "attention workspace allocation failed");
    c->ws_bytes = p.total;
    *ctx = hold.release();
    return OC_OK;
}

int oc_context_create(int device, const oc_kv_pool *kv_pool, const oc_pipeline_opts *opts, int64_t max_prefix_tokens,
                      int64_t max_suffix_tokens, void **ctx) {
    return guarded([&] {
        return context_create_body(device, kv_pool, opts, max_prefix_tokens, max_suffix_tokens, ctx);
    });
}

static int pipeline_run_body(void *ctx, const oc_request *reqs, int32_t n_reqs, oc_request_stats *stats) {
    clear_error();
    Context *c = static_cast<Context *>(ctx);
    if (!c || !reqs || n_reqs < 1) return fail(OC_EINVAL, "NULL context/requests or n_reqs < 1");
    int rc = validate_requests(c, reqs, n_reqs);
    if (rc) return rc;
    return run_pipeline(c, reqs, n_reqs, stats);
}

int oc_pipeline_run(void *ctx, const oc_request *reqs, int32_t n_reqs, oc_request_stats *stats) {
    return guarded([&] { return pipeline_run_body(ctx, reqs, n_reqs, stats); });
}

double oc_pipeline_last_ms(void *ctx) { return ctx ? static_cast<Context *>(ctx)->last_ms : 0.0; }

void oc_context_destroy(void *ctx) { release(static_cast<Context *>(ctx)); }

}  // extern "C"

// pcs_runtime.cpp -- host runtime behind the C ABI in include/pcs.h.
//
// Owns: the arena sub-allocator (first fit over a caller-owned device
// arena), the snapshot table (handle -> immutable snapshot record, shared by
// forks, kept alive by incremental children), the descriptor builder (plan
// buffers -> logical/physical runs and 64-chunk groups), pinned staging for
// descriptor uploads, and stream ordering.  Every byte of state moves in the
// kernels of pcs_kernels.hip; nothing here touches snapshot data on the host.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/pcs.h"
#include "pcs_device.h"
#include "pcs_host.h"

namespace pcs {
namespace {

constexpr uint64_t kMaxGroups = (1ULL << 32) / 256 - 1;  // grid limit of the 256-lane kernels
constexpr uint32_t kStagingSlots = 8;
constexpr uint32_t kCountPairs = 2048;  // host word pairs (stored-chunk count, payload top), pair 0 for exact calls
// A new segment for incremental payloads takes this share of the largest
// free block (at least the call's worst case).
constexpr uint64_t kSegmentShareNum = 1, kSegmentShareDen = 2;
// Limits of pcs_fingerprint_noalloc: its descriptor tables pass through one
// pinned host buffer of kNoAllocStagingBytes made at context creation.
constexpr uint32_t kNoAllocMaxBufs = 4096, kNoAllocMaxRuns = 65536;
constexpr uint64_t kNoAllocStagingBytes = 2ULL << 20;
constexpr int kMaxDevices = 64;

struct SnapNode;

// A block of the arena whose incremental payload slots the device places
// downwards from `hi` (a bump word the scan kernels advance in stream
// order), so the payloads of consecutive calls lie next to each other.  The
// host claims each pending call's worst case (one slot per chunk) against it
// and, once the call's stored-chunk count is read, only its actual slots.
// The unused low part [lo, fill) goes back to the arena as soon as no call
// placed here is pending; the segment is then closed.
struct Segment {
    uint64_t lo = 0, hi = 0;
    uint64_t claim = 0;    // bytes below hi: settled calls' slots + pending calls' worst cases
    uint64_t fill = 0;     // lowest slot placed by a settled call (hi before any)
    uint32_t pending = 0;  // calls placed here whose count is not read yet
    bool started = false;  // a call has set the bump word to hi
    bool open = true;      // new calls may use it
    bool retired = false;  // its unused part went back to the arena
};

// An incremental checkpoint enqueued on the stream whose stored-chunk count
// the host has not read yet.  It outlives its snapshot if that is deleted
// first (then the slots are released when the count arrives).
struct PendingCall {
    std::weak_ptr<SnapNode> node;
    std::shared_ptr<Segment> seg;
    uint64_t worst = 0;      // bytes claimed in the segment until settled
    uint32_t pair = 0;       // host words 2*pair (count) and 2*pair+1 (top)
    hipEvent_t ev = nullptr; // recorded after the call's last kernel
};

}  // namespace
}  // namespace pcs

struct pcs_ctx {
    uint64_t arena_dev = 0;    // 4096-aligned device address of arena offset 0
    hipStream_t stream = nullptr;
    pcs::Arena arena;
    std::unordered_map<uint64_t, std::shared_ptr<pcs::SnapNode>> handles;
    uint64_t next_handle = 1;
    std::string err;

    struct Slot {
        void *host = nullptr;
        size_t cap = 0;
        hipEvent_t ev = nullptr;
        bool pending = false;
    } staging[pcs::kStagingSlots];
    uint32_t next_slot = 0;

    uint64_t *counts = nullptr;              // pinned word pairs, one per pending incremental checkpoint
    uint64_t *counts_dev = nullptr;          // the same words as the device addresses them
    std::vector<uint32_t> free_pairs;
    std::deque<pcs::PendingCall> pending;    // in stream order
    std::shared_ptr<pcs::Segment> seg;       // the open segment, if any
    hipEvent_t exact_ev = nullptr;           // an exact-size incremental call waits on it

    // The arena's first unit, kept by the library: words 0 and 2 are the bump
    // words of incremental slot placement (a call reads word bump_par and
    // writes the other, which the next call reads), word 1 a call's payload
    // top.
    uint64_t bump_dev = 0, top_dev = 0;
    uint32_t bump_par = 0;

    pcs::TileDevice dev{0, 0};  // CU count and real-time counter rate of the arena's device (0: unknown)

    int timing = PCS_TIMING_OFF;  // pcs_set_timing mode
    bool no_events = false;  // set while a call that must create nothing runs (no timing events)
    std::map<std::string, std::vector<std::pair<hipEvent_t, hipEvent_t>>> timers;

    // pcs_fingerprint_noalloc: the device's static scratch array (its address
    // on the arena's device) and a fixed pinned staging buffer for tables.
    uint64_t scratch_dev = 0;
    void *na_host = nullptr;
    hipEvent_t na_ev = nullptr;
    bool na_pending = false;
};

namespace pcs {
namespace {

struct SnapNode {
    pcs_ctx *ctx = nullptr;
    uint64_t block_off = 0, block_bytes = 0;
    uint32_t nbufs = 0;
    bool incremental = false, has_hashes = false;
    std::vector<Layout> bufs;
    std::vector<uint64_t> chunk_begin;  // per buffer, in this snapshot's chunk order
    std::vector<uint64_t> comp_off;     // full: component offset inside the payload
    uint64_t total_chunks = 0, state_bytes = 0;
    uint64_t hashes_off = 0, manifest_off = 0, roots_off = 0, payload_off = 0;  // arena offsets
    uint64_t payload_bytes = 0;         // stored bytes (incremental: after settling)
    uint64_t pay_off = 0, pay_bytes = 0;  // incremental: its slots (known once settled)
    uint64_t pay_top = 0;               // incremental: arena offset of the top of its slots
    bool settled = true;                // incremental: stored-chunk count read
    std::shared_ptr<SnapNode> parent;   // chunks this snapshot's manifest points into

    ~SnapNode()
    {
        if (block_bytes) ctx->arena.release(block_off, block_bytes);
        // An unsettled snapshot's slots are released by its pending call.
        if (settled && pay_bytes) ctx->arena.release(pay_off, pay_bytes);
    }
};

int fail(pcs_ctx *c, int code, const char *fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(pcs_ctx *c, int code, const char *fmt, ...)
{
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        c->err = buf;
    }
    return code;
}

int hip_fail(pcs_ctx *c, hipError_t e, const char *what)
{
    return fail(c, PCS_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(ctx, expr)                                              \
    do {                                                                \
        hipError_t e_ = (expr);                                         \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr);        \
    } while (0)

// Validates one descriptor and appends its runs (see pcs::describe); the
// reason for a rejection becomes the context's last error.
int check_buf(pcs_ctx *c, const pcs_buf &b, uint32_t idx, Layout *lay, std::vector<Run> *runs)
{
    std::string why;
    const int st = describe(b, idx, lay, runs, &why);
    return st ? fail(c, st, "%s", why.c_str()) : PCS_OK;
}

// A job under construction: buffer table, run table, and group totals.
struct Job {
    std::vector<JobBuf> bufs;
    std::vector<Run> runs;
    std::vector<Layout> lays;
    uint64_t ngroups = 0, nchunks = 0;
};

int add_buffers(pcs_ctx *c, Job &job, const pcs_buf *bufs, uint32_t n, uint32_t idx0)
{
    for (uint32_t i = 0; i < n; ++i) {
        Layout lay;
        const size_t r0 = job.runs.size();
        const int st = check_buf(c, bufs[i], idx0 + i, &lay, &job.runs);
        if (st) return st;
        if (job.runs.size() > (1ULL << 31)) return fail(c, PCS_E_INVAL, "too many runs");
        JobBuf jb{};
        jb.nbytes = lay.nbytes;
        jb.nchunks = lay.nchunks;
        jb.chunk_begin = job.nchunks;
        jb.group_begin = job.ngroups;
        jb.run_begin = (uint32_t)r0;
        jb.run_count = (uint32_t)(job.runs.size() - r0);
        job.nchunks += lay.nchunks;
        job.ngroups += lay.ngroups;
        if (job.ngroups > kMaxGroups) return fail(c, PCS_E_INVAL, "job too large (%llu groups)", (unsigned long long)job.ngroups);
        job.bufs.push_back(jb);
        job.lays.push_back(lay);
    }
    return PCS_OK;
}

// Per-call device scratch from the arena, released when the call returns.
// Reuse is safe: later users are stream-ordered after this call's kernels.
struct Temp {
    pcs_ctx *c;
    uint64_t off = 0, bytes = 0;
    explicit Temp(pcs_ctx *ctx) : c(ctx) {}
    ~Temp()
    {
        if (bytes) c->arena.release(off, bytes);
    }
    Temp(const Temp &) = delete;
    Temp &operator=(const Temp &) = delete;
};

// Carves sub-buffers out of one temp block.
struct Carver {
    std::vector<std::pair<uint64_t *, uint64_t>> parts;  // (where to store offset, bytes)
    uint64_t total = 0;
    void add(uint64_t *off, uint64_t bytes)
    {
        *off = total;
        total += round_up(std::max<uint64_t>(bytes, 8), 256);
    }
};

int temp_alloc(pcs_ctx *c, Temp &t, uint64_t bytes)
{
    if (!c->arena.alloc(bytes, &t.off))
        return fail(c, PCS_E_NOMEM, "arena cannot hold %llu bytes of scratch", (unsigned long long)bytes);
    t.bytes = bytes;
    return PCS_OK;
}

// Copies host bytes to device memory through a pinned staging slot.
int upload(pcs_ctx *c, uint64_t dev, const void *src, size_t bytes)
{
    if (bytes == 0) return PCS_OK;
    pcs_ctx::Slot &s = c->staging[c->next_slot];
    c->next_slot = (c->next_slot + 1) % kStagingSlots;
    if (s.pending) {
        HIP_TRY(c, hipEventSynchronize(s.ev));
        s.pending = false;
    }
    if (s.cap < bytes) {
        if (s.host) HIP_TRY(c, hipHostFree(s.host));
        s.host = nullptr;
        const size_t cap = round_up(bytes, 1 << 20);
        HIP_TRY(c, hipHostMalloc(&s.host, cap, hipHostMallocDefault));
        s.cap = cap;
    }
    memcpy(s.host, src, bytes);
    HIP_TRY(c, hipMemcpyAsync((void *)dev, s.host, bytes, hipMemcpyHostToDevice, c->stream));
    HIP_TRY(c, hipEventRecord(s.ev, c->stream));
    s.pending = true;
    return PCS_OK;
}

template <class F>
int launch(pcs_ctx *c, const char *name, F &&f)
{
    hipEvent_t a = nullptr, b = nullptr;
    auto drop = [&] {
        if (a) (void)hipEventDestroy(a);
        if (b) (void)hipEventDestroy(b);
    };
    // PCS_TIMING_EVENTS records the pair on the stream around the launcher's
    // launch; PCS_TIMING_DISPATCH hands it to the kernel launch itself, which
    // stamps the kernel's own begin and end (a launcher with no work launches
    // nothing, and the pair is then recorded back to back: zero time).
    const bool timed = c->timing != PCS_TIMING_OFF && !c->no_events;
    const bool dispatch = c->timing == PCS_TIMING_DISPATCH;
    if (timed) {
        hipError_t te = hipEventCreate(&a);
        if (te == hipSuccess) te = hipEventCreate(&b);
        if (te == hipSuccess && !dispatch) te = hipEventRecord(a, c->stream);
        if (te != hipSuccess) {
            drop();
            return hip_fail(c, te, "timing event");
        }
        if (dispatch) set_kernel_events(a, b);
    }
    const hipError_t e = f();
    if (timed) {
        hipError_t te = hipSuccess;
        if (!dispatch) {
            te = hipEventRecord(b, c->stream);
        } else if (!take_kernel_events_used()) {
            te = hipEventRecord(a, c->stream);
            if (te == hipSuccess) te = hipEventRecord(b, c->stream);
        }
        if (te != hipSuccess || e != hipSuccess) {
            drop();
            return e != hipSuccess ? hip_fail(c, e, name) : hip_fail(c, te, "timing event");
        }
        c->timers[name].push_back({a, b});
    }
    if (e != hipSuccess) return hip_fail(c, e, name);
    return PCS_OK;
}

// Retires a segment no pending call uses any more: its unused low part goes
// back to the arena, and it takes no new calls.
void retire_if_idle(pcs_ctx *c, const std::shared_ptr<Segment> &g)
{
    if (g->pending || g->retired) return;
    if (g->fill > g->lo) c->arena.release(g->lo, g->fill - g->lo);
    g->retired = true;
    g->open = false;
    if (c->seg == g) c->seg.reset();
}

// Reads a finished call's stored-chunk count and payload top: the snapshot
// learns where its slots are, the segment's claim drops to the actual slots.
void finish_call(pcs_ctx *c, PendingCall &p)
{
    const uint64_t dirty = c->counts[2 * p.pair], top = c->counts[2 * p.pair + 1];
    const uint64_t bytes = dirty * kChunk;
    c->free_pairs.push_back(p.pair);
    (void)hipEventDestroy(p.ev);
    p.ev = nullptr;
    Segment &g = *p.seg;
    g.claim = g.claim - p.worst + bytes;
    g.fill = top - bytes;
    --g.pending;
    if (auto n = p.node.lock()) {
        n->pay_off = n->payload_off = top - bytes;
        n->pay_bytes = n->payload_bytes = bytes;
        n->pay_top = top;
        n->settled = true;
    } else if (bytes) {
        c->arena.release(top - bytes, bytes);  // deleted before its count arrived
    }
    retire_if_idle(c, p.seg);
}

// Settles pending calls in stream order: those already finished, or (wait)
// every one, waiting for each.  Stops at the first that has not finished or
// whose wait failed.
void settle(pcs_ctx *c, bool wait)
{
    while (!c->pending.empty()) {
        PendingCall &p = c->pending.front();
        const hipError_t q = wait ? hipEventSynchronize(p.ev) : hipEventQuery(p.ev);
        if (q != hipSuccess) return;
        finish_call(c, p);
        c->pending.pop_front();
    }
}

// Waits for the oldest pending call and settles it (and every other one
// that has finished).  False if none is pending or the wait failed, so that
// callers never retry without progress.
bool settle_oldest(pcs_ctx *c)
{
    if (c->pending.empty()) return false;
    PendingCall &p = c->pending.front();
    if (hipEventSynchronize(p.ev) != hipSuccess) return false;
    finish_call(c, p);
    c->pending.pop_front();
    settle(c, false);
    return true;
}

// Allocates a snapshot block (from the bottom, or the top of the arena),
// first settling finished incremental checkpoints, then waiting for pending
// ones oldest first until the block fits: the wait ends as soon as enough
// space has come back (a segment closes when its last pending call is
// settled), not when the stream is idle.
bool alloc_settled(pcs_ctx *c, uint64_t bytes, uint64_t *off, bool top)
{
    auto try_alloc = [&] { return top ? c->arena.alloc_top(bytes, off) : c->arena.alloc(bytes, off); };
    settle(c, false);
    if (try_alloc()) return true;
    while (settle_oldest(c))
        if (try_alloc()) return true;
    return false;
}

// The segment an incremental call of worst case `worst` bytes is placed in:
// the open one if its unclaimed part holds the worst case, else a new one of
// max(worst, half the largest free block) from the top of the arena (the old
// one then closes once its pending calls settle), waiting for pending calls
// oldest first while neither fits.  Null if nothing fits with no call
// pending: the call then takes the exact path.
std::shared_ptr<Segment> segment_for(pcs_ctx *c, uint64_t worst)
{
    settle(c, false);
    for (;;) {
        const auto &g = c->seg;
        if (g && g->open && worst <= g->hi - g->lo - g->claim) return g;
        const uint64_t share = c->arena.largest() / kSegmentShareDen * kSegmentShareNum / kAlign * kAlign;
        const uint64_t size = std::max(worst, share);
        uint64_t off = 0;
        if (c->arena.largest() >= size && c->arena.alloc_top(size, &off)) {
            auto ng = std::make_shared<Segment>();
            ng->lo = off;
            ng->hi = ng->fill = off + round_up(size, kAlign);
            if (c->seg) {
                auto old = c->seg;
                old->open = false;
                c->seg.reset();
                retire_if_idle(c, old);  // now, or when its last pending call settles
            }
            c->seg = ng;
            return ng;
        }
        if (!settle_oldest(c)) return nullptr;
    }
}

bool alloc_block(pcs_ctx *c, uint64_t bytes, uint64_t *off) { return alloc_settled(c, bytes, off, false); }
bool alloc_block_top(pcs_ctx *c, uint64_t bytes, uint64_t *off) { return alloc_settled(c, bytes, off, true); }

std::shared_ptr<SnapNode> lookup(pcs_ctx *c, pcs_snap h)
{
    auto it = c->handles.find(h);
    return it == c->handles.end() ? nullptr : it->second;
}

pcs_snap new_handle(pcs_ctx *c, std::shared_ptr<SnapNode> n)
{
    const pcs_snap h = c->next_handle++;
    c->handles.emplace(h, std::move(n));
    return h;
}

// Shared part of fingerprint / full checkpoint / batch checkpoint: a job over
// `sessions` sessions whose buffers are already in `job`; fingerprints of
// buffer b go to job.bufs[b].hash_dst, roots to root_dst[b][0..1], session
// roots to sroot_dst[s][0..1].
struct RootDst {
    uint64_t d[2];
};

bool is_small(const Job &job) { return job.bufs.size() <= kArgBufs && job.runs.size() <= kArgRuns; }

// The descriptor tables of a job as the kernels see them: in the kernel
// arguments for a small job, else uploaded into per-call scratch with a
// group -> buffer map.
struct Staged {
    bool small = false;
    ArgTables arg;
    DevTables dev;
};

// Lays out per-call scratch as [tables (big jobs)][extra host bytes] (one
// upload) then [group map (big jobs)][dev_bytes of device-only scratch],
// uploads, and launches the group map for a big job.
int stage(pcs_ctx *c, const Job &job, bool small, Temp &t, const std::vector<uint8_t> &extra, uint64_t dev_bytes,
          Staged &sg, uint64_t &extra_dev, uint64_t &scratch_dev)
{
    const uint32_t n = (uint32_t)job.bufs.size();
    const uint64_t G = job.ngroups;
    Carver cv;
    uint64_t o_bufs = 0, o_runs = 0, o_extra = 0, o_map = 0, o_scr = 0;
    if (!small) {
        cv.add(&o_bufs, sizeof(JobBuf) * n);
        cv.add(&o_runs, sizeof(Run) * job.runs.size());
    }
    if (!extra.empty()) cv.add(&o_extra, extra.size());
    const uint64_t hb = cv.total;
    if (!small) cv.add(&o_map, sizeof(GroupRef) * G);
    if (dev_bytes) cv.add(&o_scr, dev_bytes);
    // A small job with nothing to upload and no device scratch (a restore,
    // a plain pack, classify) takes no arena space at all.
    uint64_t base = 0;
    if (cv.total) {
        if (int e = temp_alloc(c, t, cv.total)) return e;
        base = c->arena_dev + t.off;
    }
    extra_dev = extra.empty() ? 0 : base + o_extra;
    scratch_dev = dev_bytes ? base + o_scr : 0;
    sg.small = small;
    if (small) {
        memset(&sg.arg, 0, sizeof sg.arg);
        sg.arg.nbuf = n;
        if (n) memcpy(sg.arg.bufs, job.bufs.data(), sizeof(JobBuf) * n);
        if (!job.runs.empty()) memcpy(sg.arg.runs, job.runs.data(), sizeof(Run) * job.runs.size());
    } else {
        sg.dev = DevTables{(const JobBuf *)(base + o_bufs), (const Run *)(base + o_runs),
                           (const GroupRef *)(base + o_map), n, 0};
    }
    if (hb) {
        std::vector<uint8_t> host(hb, 0);
        if (!small) {
            if (n) memcpy(host.data() + o_bufs, job.bufs.data(), sizeof(JobBuf) * n);
            if (!job.runs.empty()) memcpy(host.data() + o_runs, job.runs.data(), sizeof(Run) * job.runs.size());
        }
        if (!extra.empty()) memcpy(host.data() + o_extra, extra.data(), extra.size());
        if (int e = upload(c, base, host.data(), hb)) return e;
    }
    if (!small && G)
        return launch(c, "map", [&] {
            return launch_group_map(sg.dev.bufs, sg.dev.runs, n, G, (GroupRef *)sg.dev.map, c->stream);
        });
    return PCS_OK;
}

template <class F>
int with_tables(const Staged &sg, F &&f)
{
    return sg.small ? f(sg.arg) : f(sg.dev);
}

std::vector<uint8_t> bytes_of(const std::vector<MerkleList> &lists)
{
    std::vector<uint8_t> v(sizeof(MerkleList) * lists.size());
    if (!lists.empty()) memcpy(v.data(), lists.data(), v.size());
    return v;
}

ArgLists arg_lists(const std::vector<MerkleList> &lists, uint32_t nbuf_lists)
{
    ArgLists al;
    memset(&al, 0, sizeof al);
    al.nbuf_lists = nbuf_lists;
    al.nlists = (uint32_t)lists.size();
    for (size_t j = 0; j < lists.size(); ++j) al.lists[j] = lists[j];
    return al;
}

// Buffer roots then session roots: one single-workgroup launch for a small
// job, else one workgroup per list in two launches.  Buffer lists of more
// than kMerkleLdsValues values (up to kLongLists of them) first have their
// 64-value blocks reduced by every CU (one more launch), which a single
// workgroup would otherwise do a block per wavefront at a time.
int run_merkle(pcs_ctx *c, bool small, const std::vector<MerkleList> &lists, uint32_t nbuf_lists,
               uint64_t lists_dev, uint64_t *d_nodes, uint64_t *d_sa, uint64_t *d_sb, uint64_t *d_roots)
{
    hipStream_t s = c->stream;
    LongLists ll{};
    uint32_t nlong = 0;
    for (uint32_t j = 0; j < nbuf_lists; ++j)
        if (lists[j].count > kMerkleLdsValues) {
            if (nlong < kLongLists) {
                ll.begin[nlong] = lists[j].begin;
                ll.count[nlong] = lists[j].count;
                ll.block_begin[nlong + 1] = ll.block_begin[nlong] + (lists[j].count + 63) / 64;
            }
            ++nlong;
        }
    const bool pre = nlong > 0 && nlong <= kLongLists;
    if (pre) {
        ll.n = nlong;
        if (int st = launch(c, "merkle", [&] { return launch_merkle_blocks(ll, d_nodes, d_sa, s); })) return st;
    }
    if (small) {
        const ArgLists al = arg_lists(lists, nbuf_lists);
        return launch(c, "merkle", [&] { return launch_merkle_small(al, d_nodes, d_sa, d_sb, pre, s); });
    }
    const MerkleList *d_lists = (const MerkleList *)lists_dev;
    const uint32_t nsess = (uint32_t)lists.size() - nbuf_lists;
    uint64_t max_buf = 0, max_sess = 0;  // the longest list of each launch picks its workgroup size
    for (size_t j = 0; j < lists.size(); ++j) {
        uint64_t &m = j < nbuf_lists ? max_buf : max_sess;
        m = std::max(m, lists[j].count);
    }
    if (int st = launch(c, "merkle", [&] {
            return launch_merkle(d_lists, nbuf_lists, d_nodes, d_sa, d_sb, d_roots, max_buf, pre, s);
        }))
        return st;
    return launch(c, "merkle", [&] {
        return launch_merkle(d_lists + nbuf_lists, nsess, d_roots, d_sa, d_sb, nullptr, max_sess, false, s);
    });
}

int run_hash_job(pcs_ctx *c, Job &job, bool copy, const std::vector<uint32_t> &sess_nbufs,
                 const std::vector<RootDst> &root_dst, const std::vector<RootDst> &sroot_dst,
                 bool want_roots)
{
    const uint32_t n = (uint32_t)job.bufs.size();
    const uint32_t S = (uint32_t)sess_nbufs.size();
    const uint64_t G = job.ngroups;
    const bool small = is_small(job) && S <= 1;
    // A small job runs as sub-tiles: one Merkle node per sub-tile, and each
    // buffer's list covers its sub-tiles (aligned subtrees of the same tree).
    const uint32_t tiles = tile_split(G);
    const uint64_t per_tile = kGroupChunks / tiles;
    std::vector<MerkleList> lists;
    if (want_roots) {
        for (uint32_t b = 0; b < n; ++b)
            lists.push_back({job.bufs[b].group_begin * tiles, div_up(job.bufs[b].nchunks, per_tile),
                             {root_dst[b].d[0], root_dst[b].d[1]}});
        uint64_t first = 0;
        for (uint32_t s = 0; s < S; ++s) {
            lists.push_back({first, sess_nbufs[s], {sroot_dst[s].d[0], sroot_dst[s].d[1]}});
            first += sess_nbufs[s];
        }
    }
    Carver cv;
    uint64_t o_nodes, o_sa, o_sb, o_roots;
    cv.add(&o_nodes, 8 * G * tiles);
    cv.add(&o_sa, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_sb, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_roots, 8 * n);
    Temp t(c);
    Staged sg;
    uint64_t lists_dev, scr;
    if (int st = stage(c, job, small, t, small ? std::vector<uint8_t>() : bytes_of(lists), cv.total, sg, lists_dev, scr))
        return st;
    uint64_t *d_nodes = (uint64_t *)(scr + o_nodes);
    uint64_t *d_sa = (uint64_t *)(scr + o_sa), *d_sb = (uint64_t *)(scr + o_sb);
    uint64_t *d_roots = (uint64_t *)(scr + o_roots);
    hipStream_t s = c->stream;
    int st = with_tables(sg, [&](const auto &tab) {
        return launch(c, copy ? "pack_hash" : "hash", [&] {
            return launch_tile(tab, G, copy ? kModePack : kModeHash, d_nodes, nullptr, 0, s, tiles, c->dev);
        });
    });
    if (st || !want_roots) return st;
    return run_merkle(c, small, lists, n, lists_dev, d_nodes, d_sa, d_sb, d_roots);
}

struct FullPlan {
    std::vector<uint64_t> comp_off;
    uint64_t payload = 0, hashes_rel = 0, roots_rel = 0, payload_rel = 0, block = 0;
};

FullPlan full_plan(const Job &job, size_t b0, size_t nb, uint64_t nchunks, bool hashes)
{
    FullPlan p;
    for (size_t b = b0; b < b0 + nb; ++b) {
        p.comp_off.push_back(p.payload);
        p.payload += job.lays[b].nchunks * kChunk;
    }
    uint64_t off = 0;
    p.hashes_rel = off;
    if (hashes) off += 8 * nchunks;
    p.roots_rel = off;
    off += 8 * (nb + 1);
    p.payload_rel = round_up(off, kAlign);
    p.block = p.payload_rel + p.payload;
    return p;
}

std::shared_ptr<SnapNode> make_node(pcs_ctx *c, const Job &job, size_t b0, size_t nb, const FullPlan &p,
                                    uint64_t block_off, bool hashes)
{
    auto node = std::make_shared<SnapNode>();
    node->ctx = c;
    node->block_off = block_off;
    node->block_bytes = p.block;
    node->nbufs = (uint32_t)nb;
    node->has_hashes = hashes;
    uint64_t cb = 0;
    for (size_t b = b0; b < b0 + nb; ++b) {
        node->bufs.push_back(job.lays[b]);
        node->chunk_begin.push_back(cb);
        cb += job.lays[b].nchunks;
        node->state_bytes += job.lays[b].nbytes;
    }
    node->total_chunks = cb;
    node->comp_off = p.comp_off;
    node->hashes_off = block_off + p.hashes_rel;
    node->roots_off = block_off + p.roots_rel;
    node->payload_off = block_off + p.payload_rel;
    node->payload_bytes = p.payload;
    return node;
}

// Full checkpoints of several sessions in one launch.
int checkpoint_full(pcs_ctx *c, const pcs_buf *plans, const uint32_t *nbufs, uint32_t sessions, uint32_t flags,
                    uint64_t *d_hashes, uint64_t *d_roots, uint64_t *d_sroots, pcs_snap *out)
{
    const bool hash = (flags & PCS_CKPT_HASH) != 0;
    if (!hash && (d_hashes || d_roots || d_sroots))
        return fail(c, PCS_E_INVAL, "fingerprint outputs need PCS_CKPT_HASH");
    Job job;
    uint64_t nb_total = 0;
    for (uint32_t s = 0; s < sessions; ++s) nb_total += nbufs[s];
    if (nb_total > (1u << 24)) return fail(c, PCS_E_INVAL, "too many buffers");
    if (int st = add_buffers(c, job, plans, (uint32_t)nb_total, 0)) return st;

    // Reserve every snapshot block first (all or none).
    std::vector<FullPlan> fps;
    std::vector<uint64_t> offs;
    size_t b0 = 0;
    for (uint32_t s = 0; s < sessions; ++s) {
        uint64_t nch = 0;
        for (size_t b = b0; b < b0 + nbufs[s]; ++b) nch += job.lays[b].nchunks;
        fps.push_back(full_plan(job, b0, nbufs[s], nch, hash));
        uint64_t off;
        if (!alloc_block(c, fps.back().block, &off)) {
            for (size_t k = 0; k < offs.size(); ++k) c->arena.release(offs[k], fps[k].block);
            return fail(c, PCS_E_NOMEM, "arena cannot hold snapshot %u (%llu bytes)", s,
                        (unsigned long long)fps.back().block);
        }
        offs.push_back(off);
        b0 += nbufs[s];
    }
    std::vector<std::shared_ptr<SnapNode>> nodes;
    b0 = 0;
    for (uint32_t s = 0; s < sessions; ++s) {
        nodes.push_back(make_node(c, job, b0, nbufs[s], fps[s], offs[s], hash));
        b0 += nbufs[s];
    }

    // Wire destinations.
    std::vector<RootDst> rdst(nb_total), sdst(sessions);
    b0 = 0;
    uint64_t chunk0 = 0;
    for (uint32_t s = 0; s < sessions; ++s) {
        const auto &nd = nodes[s];
        for (uint32_t k = 0; k < nbufs[s]; ++k) {
            JobBuf &jb = job.bufs[b0 + k];
            jb.payload = c->arena_dev + nd->payload_off + nd->comp_off[k];
            if (hash) {
                jb.hash_dst[0] = c->arena_dev + nd->hashes_off + 8 * nd->chunk_begin[k];
                jb.hash_dst[1] = d_hashes ? (uint64_t)(d_hashes + jb.chunk_begin) : 0;
                rdst[b0 + k].d[0] = c->arena_dev + nd->roots_off + 8 * k;
                rdst[b0 + k].d[1] = d_roots ? (uint64_t)(d_roots + b0 + k) : 0;
            }
        }
        sdst[s].d[0] = c->arena_dev + nd->roots_off + 8 * nbufs[s];
        sdst[s].d[1] = d_sroots ? (uint64_t)(d_sroots + s) : 0;
        b0 += nbufs[s];
        chunk0 += nd->total_chunks;
    }
    (void)chunk0;

    int st;
    if (hash) {
        std::vector<uint32_t> sn(nbufs, nbufs + sessions);
        st = run_hash_job(c, job, true, sn, rdst, sdst, true);
    } else {
        Temp t(c);
        Staged sg;
        uint64_t xd, scr;
        st = stage(c, job, is_small(job), t, {}, 0, sg, xd, scr);
        const uint64_t G = job.ngroups;
        if (!st)
            st = with_tables(sg, [&](const auto &tab) {
                return launch(c, "pack", [&] { return launch_copy(tab, G, true, 0, c->stream, c->dev.cus); });
            });
    }
    if (st) return st;  // nodes (and their blocks) are released here
    for (uint32_t s = 0; s < sessions; ++s) out[s] = new_handle(c, nodes[s]);
    return PCS_OK;
}

// strict: a destination must have the snapshot buffer's kind and ring shape;
// otherwise only its logical size must match (used to lay a snapshot out
// flat, e.g. for export).
int restore_impl(pcs_ctx *c, const pcs_snap *snaps, uint32_t m, const pcs_buf *dsts, const uint32_t *nbufs,
                 bool strict)
{
    if (!c) return PCS_E_INVAL;
    if (m && (!snaps || !nbufs)) return fail(c, PCS_E_INVAL, "null argument");
    Job job;
    uint64_t nb_total = 0;
    std::vector<std::shared_ptr<SnapNode>> nodes;
    for (uint32_t j = 0; j < m; ++j) {
        auto nd = lookup(c, snaps[j]);
        if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snaps[j]);
        if (nbufs[j] != nd->nbufs)
            return fail(c, PCS_E_SHAPE, "snapshot %u holds %u buffers, %u destinations given", j, nd->nbufs, nbufs[j]);
        nodes.push_back(nd);
        nb_total += nbufs[j];
    }
    if (nb_total && !dsts) return fail(c, PCS_E_INVAL, "null destinations");
    if (nb_total > (1u << 24)) return fail(c, PCS_E_INVAL, "too many buffers");
    if (int st = add_buffers(c, job, dsts, (uint32_t)nb_total, 0)) return st;
    uint32_t b = 0;
    for (uint32_t j = 0; j < m; ++j) {
        const auto &nd = nodes[j];
        for (uint32_t k = 0; k < nd->nbufs; ++k, ++b) {
            const Layout &want = nd->bufs[k], &got = job.lays[b];
            if (want.nbytes != got.nbytes ||
                (strict && (want.kind != got.kind ||
                            (want.kind == PCS_RING && (want.row_bytes != got.row_bytes ||
                                                       want.window != got.window || want.outer != got.outer)))))
                return fail(c, PCS_E_SHAPE, "restore %u buffer %u: destination layout differs from the snapshot", j, k);
            JobBuf &jb = job.bufs[b];
            if (nd->incremental)
                jb.manifest = c->arena_dev + nd->manifest_off + 8 * nd->chunk_begin[k];
            else
                jb.payload = c->arena_dev + nd->payload_off + nd->comp_off[k];
        }
    }
    const uint32_t n = (uint32_t)nb_total;
    if (n == 0) return PCS_OK;
    Temp t(c);
    Staged sg;
    uint64_t xd, scr;
    if (int st = stage(c, job, is_small(job), t, {}, 0, sg, xd, scr)) return st;
    const uint64_t G = job.ngroups;
    return with_tables(sg, [&](const auto &tab) {
        return launch(c, "copy", [&] { return launch_copy(tab, G, false, c->arena_dev, c->stream); });
    });
}


// Fingerprints flat device regions (e.g. payload components) into device
// arrays: chunk hashes (buffer-major), buffer roots, session root.
int fingerprint_regions(pcs_ctx *c, const std::vector<uint64_t> &addr, const std::vector<uint64_t> &nbytes,
                        uint64_t *d_hashes, uint64_t *d_roots, uint64_t *d_sroot)
{
    const uint32_t n = (uint32_t)addr.size();
    std::vector<pcs_buf> bufs(n);
    for (uint32_t b = 0; b < n; ++b) {
        memset(&bufs[b], 0, sizeof(pcs_buf));
        bufs[b].ptr = addr[b];
        bufs[b].nbytes = nbytes[b];
        bufs[b].kind = PCS_FLAT;
    }
    Job job;
    if (int st = add_buffers(c, job, bufs.data(), n, 0)) return st;
    std::vector<RootDst> rdst(n), sdst(1);
    for (uint32_t b = 0; b < n; ++b) {
        job.bufs[b].hash_dst[0] = (uint64_t)(d_hashes + job.bufs[b].chunk_begin);
        rdst[b].d[0] = (uint64_t)(d_roots + b);
    }
    sdst[0].d[0] = (uint64_t)d_sroot;
    return run_hash_job(c, job, false, {n}, rdst, sdst, true);
}

// The static scratch array's address on the device that holds `dev_ptr`,
// looked up once per device (with that device current) and kept for the
// life of the process: each GPU holds its own copy at its own address.
hipError_t scratch_for(const void *dev_ptr, uint64_t *addr)
{
    static std::mutex mu;
    static uint64_t cached[kMaxDevices];
    hipPointerAttribute_t at;
    hipError_t e = hipPointerGetAttributes(&at, dev_ptr);
    if (e != hipSuccess) return e;
    const int dev = at.device;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!cached[dev]) {
        int cur = 0;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        uint64_t a = 0;
        e = static_scratch_address(&a);
        const hipError_t back = cur != dev ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess) return e;
        if (back != hipSuccess) return back;
        cached[dev] = a;
    }
    *addr = cached[dev];
    return hipSuccess;
}

// Clears c->no_events when the call that set it returns.
struct NoEvents {
    pcs_ctx *c;
    explicit NoEvents(pcs_ctx *ctx) : c(ctx) { c->no_events = true; }
    ~NoEvents() { c->no_events = false; }
};

}  // namespace
}  // namespace pcs

using namespace pcs;

extern "C" {

int pcs_ctx_create(void *d_arena, uint64_t arena_bytes, void *hip_stream, pcs_ctx **out)
{
    if (!out) return PCS_E_INVAL;
    *out = nullptr;
    if (!d_arena || (uint64_t)d_arena % 16) return PCS_E_INVAL;
    const uint64_t a = (uint64_t)d_arena;
    const uint64_t aligned = round_up(a, kAlign);
    if (arena_bytes < aligned - a + 2 * kAlign) return PCS_E_INVAL;  // one unit is the library's own
    auto *c = new pcs_ctx();
    c->arena_dev = aligned;
    c->arena.init((arena_bytes - (aligned - a)) / kAlign * kAlign);
    c->stream = (hipStream_t)hip_stream;
    for (auto &s : c->staging) {
        if (hipEventCreateWithFlags(&s.ev, hipEventDisableTiming) != hipSuccess) {
            pcs_ctx_destroy(c);
            return PCS_E_HIP;
        }
    }
    if (hipHostMalloc((void **)&c->counts, 16 * kCountPairs, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
        hipHostGetDevicePointer((void **)&c->counts_dev, c->counts, 0) != hipSuccess ||
        hipEventCreateWithFlags(&c->exact_ev, hipEventDisableTiming) != hipSuccess) {
        pcs_ctx_destroy(c);
        return PCS_E_HIP;
    }
    for (uint32_t i = kCountPairs - 1; i >= 1; --i) c->free_pairs.push_back(i);  // pair 0: exact calls
    // The library's own unit: the first of the arena.
    uint64_t own = 0;
    if (!c->arena.alloc(kAlign, &own)) {
        pcs_ctx_destroy(c);
        return PCS_E_INVAL;
    }
    c->bump_dev = c->arena_dev + own;
    c->top_dev = c->bump_dev + 8;
    {
        hipPointerAttribute_t at;
        int cus = 0, khz = 0;
        if (hipPointerGetAttributes(&at, d_arena) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, at.device) == hipSuccess &&
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, at.device) == hipSuccess && cus > 0 &&
            khz > 0)
            c->dev = TileDevice{(uint32_t)cus, (uint32_t)khz};
    }
    if (hipHostMalloc(&c->na_host, kNoAllocStagingBytes, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&c->na_ev, hipEventDisableTiming) != hipSuccess ||
        scratch_for(d_arena, &c->scratch_dev) != hipSuccess) {
        pcs_ctx_destroy(c);
        return PCS_E_HIP;
    }
    *out = c;
    return PCS_OK;
}

int pcs_ctx_destroy(pcs_ctx *c)
{
    if (!c) return PCS_E_INVAL;
    (void)hipStreamSynchronize(c->stream);
    c->handles.clear();
    for (auto &p : c->pending)
        if (p.ev) (void)hipEventDestroy(p.ev);
    c->pending.clear();
    c->seg.reset();
    if (c->exact_ev) (void)hipEventDestroy(c->exact_ev);
    for (auto &kv : c->timers)
        for (auto &ab : kv.second) {
            (void)hipEventDestroy(ab.first);
            (void)hipEventDestroy(ab.second);
        }
    for (auto &s : c->staging) {
        if (s.ev) (void)hipEventDestroy(s.ev);
        if (s.host) (void)hipHostFree(s.host);
    }
    if (c->counts) (void)hipHostFree(c->counts);
    if (c->na_ev) (void)hipEventDestroy(c->na_ev);
    if (c->na_host) (void)hipHostFree(c->na_host);
    delete c;
    return PCS_OK;
}

const char *pcs_last_error(const pcs_ctx *c) { return c ? c->err.c_str() : "null context"; }

int pcs_chunk_counts(const pcs_buf *bufs, uint32_t n, uint64_t *chunks, uint64_t *total)
{
    if (n && !bufs) return PCS_E_INVAL;
    uint64_t t = 0;
    for (uint32_t i = 0; i < n; ++i) {
        Layout lay;
        std::vector<Run> rs;
        if (int st = check_buf(nullptr, bufs[i], i, &lay, &rs)) return st;
        if (chunks) chunks[i] = lay.nchunks;
        t += lay.nchunks;
    }
    if (total) *total = t;
    return PCS_OK;
}

int pcs_fingerprint(pcs_ctx *c, const pcs_buf *bufs, uint32_t n, uint64_t *d_hashes, uint64_t *d_roots,
                    uint64_t *d_sroot)
{
    if (!c) return PCS_E_INVAL;
    if (n && !bufs) return fail(c, PCS_E_INVAL, "null buffer array");
    if (n > (1u << 24)) return fail(c, PCS_E_INVAL, "too many buffers");
    Job job;
    if (int st = add_buffers(c, job, bufs, n, 0)) return st;
    std::vector<RootDst> rdst(n), sdst(1);
    for (uint32_t b = 0; b < n; ++b) {
        job.bufs[b].hash_dst[0] = d_hashes ? (uint64_t)(d_hashes + job.bufs[b].chunk_begin) : 0;
        rdst[b].d[0] = d_roots ? (uint64_t)(d_roots + b) : 0;
    }
    sdst[0].d[0] = (uint64_t)d_sroot;
    settle(c, false);
    return run_hash_job(c, job, false, {n}, rdst, sdst, d_roots || d_sroot);
}

int pcs_fingerprint_noalloc(pcs_ctx *c, const pcs_buf *bufs, uint32_t n, uint64_t *d_hashes, uint64_t *d_roots,
                            uint64_t *d_sroot)
{
    if (!c) return PCS_E_INVAL;
    if (n && !bufs) return fail(c, PCS_E_INVAL, "null buffer array");
    if (n > kNoAllocMaxBufs) return fail(c, PCS_E_INVAL, "at most %u buffers without allocation (%u given)", kNoAllocMaxBufs, n);
    if (!c->scratch_dev) return fail(c, PCS_E_HIP, "no static scratch on this device");
    Job job;
    if (int st = add_buffers(c, job, bufs, n, 0)) return st;
    if (job.runs.size() > kNoAllocMaxRuns)
        return fail(c, PCS_E_INVAL, "at most %u physical runs without allocation (%zu given)", kNoAllocMaxRuns,
                    job.runs.size());
    const uint64_t G = job.ngroups;
    const bool want_roots = d_roots || d_sroot;
    for (uint32_t b = 0; b < n; ++b) job.bufs[b].hash_dst[0] = d_hashes ? (uint64_t)(d_hashes + job.bufs[b].chunk_begin) : 0;
    const bool small = is_small(job);
    const uint32_t tiles = tile_split(G);
    const uint64_t per_tile = kGroupChunks / tiles;

    // Scratch layout: [job tables][Merkle lists] (uploaded; large jobs only),
    // [group map (large jobs)][tile nodes][two Merkle levels][buffer roots].
    std::vector<MerkleList> lists;
    Carver cv;
    uint64_t o_bufs = 0, o_runs = 0, o_lists = 0, o_map = 0, o_nodes, o_sa, o_sb, o_roots;
    if (!small) {
        cv.add(&o_bufs, sizeof(JobBuf) * n);
        cv.add(&o_runs, sizeof(Run) * job.runs.size());
        if (want_roots) cv.add(&o_lists, sizeof(MerkleList) * (n + 1));
    }
    const uint64_t hb = cv.total;
    if (!small) cv.add(&o_map, sizeof(GroupRef) * G);
    cv.add(&o_nodes, 8 * G * tiles);
    cv.add(&o_sa, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_sb, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_roots, 8 * std::max<uint32_t>(n, 1));
    if (cv.total > kStaticScratchBytes)
        return fail(c, PCS_E_INVAL, "job needs %llu bytes of scratch, more than the %llu bytes available without "
                    "allocation", (unsigned long long)cv.total, (unsigned long long)kStaticScratchBytes);
    if (hb > kNoAllocStagingBytes)
        return fail(c, PCS_E_INVAL, "job tables need %llu bytes, more than the %llu bytes of staging",
                    (unsigned long long)hb, (unsigned long long)kNoAllocStagingBytes);
    const uint64_t base = c->scratch_dev;
    uint64_t *d_nodes = (uint64_t *)(base + o_nodes);
    uint64_t *d_sa = (uint64_t *)(base + o_sa), *d_sb = (uint64_t *)(base + o_sb);
    uint64_t *d_rt = (uint64_t *)(base + o_roots);
    if (want_roots) {
        for (uint32_t b = 0; b < n; ++b)
            lists.push_back({job.bufs[b].group_begin * tiles, div_up(job.bufs[b].nchunks, per_tile),
                             {d_roots ? (uint64_t)(d_roots + b) : 0, 0}});
        lists.push_back({0, n, {(uint64_t)d_sroot, 0}});
    }
    NoEvents guard(c);
    hipStream_t s = c->stream;
    Staged sg;
    sg.small = small;
    if (small) {
        memset(&sg.arg, 0, sizeof sg.arg);
        sg.arg.nbuf = n;
        if (n) memcpy(sg.arg.bufs, job.bufs.data(), sizeof(JobBuf) * n);
        if (!job.runs.empty()) memcpy(sg.arg.runs, job.runs.data(), sizeof(Run) * job.runs.size());
    } else {
        sg.dev = DevTables{(const JobBuf *)(base + o_bufs), (const Run *)(base + o_runs),
                           (const GroupRef *)(base + o_map), n, 0};
        // The staging buffer is reused once the previous call's copy out of it has run.
        if (c->na_pending) {
            HIP_TRY(c, hipEventSynchronize(c->na_ev));
            c->na_pending = false;
        }
        uint8_t *h = (uint8_t *)c->na_host;
        memset(h, 0, hb);
        if (n) memcpy(h + o_bufs, job.bufs.data(), sizeof(JobBuf) * n);
        if (!job.runs.empty()) memcpy(h + o_runs, job.runs.data(), sizeof(Run) * job.runs.size());
        if (want_roots) memcpy(h + o_lists, lists.data(), sizeof(MerkleList) * lists.size());
        HIP_TRY(c, hipMemcpyAsync((void *)base, h, hb, hipMemcpyHostToDevice, s));
        HIP_TRY(c, hipEventRecord(c->na_ev, s));
        c->na_pending = true;
        if (G) {
            if (int st = launch(c, "map", [&] {
                    return launch_group_map(sg.dev.bufs, sg.dev.runs, n, G, (GroupRef *)sg.dev.map, s);
                }))
                return st;
        }
    }
    int st = with_tables(sg, [&](const auto &tab) {
        return launch(c, "hash", [&] { return launch_tile(tab, G, kModeHash, d_nodes, nullptr, 0, s, tiles); });
    });
    if (st || !want_roots) return st;
    return run_merkle(c, small, lists, n, base + o_lists, d_nodes, d_sa, d_sb, d_rt);
}

int pcs_classify(pcs_ctx *c, const uint64_t *d_hashes, uint32_t K, const uint64_t *h_chunks, uint32_t n,
                 uint64_t *d_bitmap, uint8_t *d_labels)
{
    if (!c) return PCS_E_INVAL;
    if (K == 0) return fail(c, PCS_E_INVAL, "K must be >= 1");
    if (n && !h_chunks) return fail(c, PCS_E_INVAL, "null chunk counts");
    if (n > (1u << 24)) return fail(c, PCS_E_INVAL, "too many buffers");
    Job job;
    for (uint32_t b = 0; b < n; ++b) {
        JobBuf jb{};
        jb.nchunks = h_chunks[b];
        jb.chunk_begin = job.nchunks;
        jb.group_begin = job.ngroups;
        job.nchunks += h_chunks[b];
        job.ngroups += div_up(h_chunks[b], kGroupChunks);
        if (job.ngroups > kMaxGroups) return fail(c, PCS_E_INVAL, "too many chunks");
        job.bufs.push_back(jb);
    }
    if (job.nchunks && !d_hashes) return fail(c, PCS_E_INVAL, "null hashes");
    if (job.ngroups && !d_bitmap) return fail(c, PCS_E_INVAL, "null bitmap");
    if (n && !d_labels) return fail(c, PCS_E_INVAL, "null labels");
    if (n == 0) return PCS_OK;
    Temp t(c);
    Staged sg;
    uint64_t xd, scr;
    if (int st = stage(c, job, is_small(job), t, {}, 0, sg, xd, scr)) return st;
    const uint64_t G = job.ngroups, T = job.nchunks;
    if (sg.small && G <= kClassifyFusedGroups)
        return launch(c, "classify", [&] {
            return launch_classify_small(sg.arg, G, d_hashes, K, T, d_bitmap, d_labels, c->stream);
        });
    return with_tables(sg, [&](const auto &tab) {
        if (int st = launch(c, "classify", [&] {
                return launch_classify(tab, G, d_hashes, K, T, d_bitmap, c->stream);
            }))
            return st;
        return launch(c, "classify", [&] { return launch_labels(tab, d_bitmap, d_labels, c->stream); });
    });
}

int pcs_keep_count(uint64_t num, uint64_t den, uint64_t n_entries, uint64_t *keep)
{
    if (!keep || den == 0 || num > den) return PCS_E_INVAL;
    if (n_entries == 0) {
        *keep = 0;
        return PCS_OK;
    }
    // n * num / den exactly (the product fits in 128 bits), rounded to the
    // nearest integer with ties to even, then at least one entry.
    const unsigned __int128 prod = (unsigned __int128)n_entries * num;
    uint64_t q = (uint64_t)(prod / den);
    const uint64_t r = (uint64_t)(prod % den);
    const unsigned __int128 twice = (unsigned __int128)r * 2;
    if (twice > den || (twice == den && (q & 1))) ++q;
    *keep = q ? q : 1;
    return PCS_OK;
}

int pcs_distance(pcs_ctx *c, const pcs_buf *bufs, uint32_t n, const uint64_t *d_ref, uint64_t *h_differing,
                 double *h_distance)
{
    if (!c) return PCS_E_INVAL;
    if (n && !bufs) return fail(c, PCS_E_INVAL, "null buffer array");
    if (n > (1u << 24)) return fail(c, PCS_E_INVAL, "too many buffers");
    Job job;
    if (int st = add_buffers(c, job, bufs, n, 0)) return st;
    const uint64_t T = job.nchunks, G = job.ngroups;
    if (T && !d_ref) return fail(c, PCS_E_INVAL, "null reference fingerprints");
    uint64_t differing = 0;
    if (T) {
        // The diff tiles compare every chunk's fingerprint with the reference
        // (a chunk the reference does not hold never occurs: same plan), one
        // mask word per group; the scan's total is the number of set bits.
        for (auto &jb : job.bufs) {
            jb.parent_hash = (uint64_t)(d_ref + jb.chunk_begin);
            jb.parent_chunks = jb.nchunks;
        }
        const uint32_t tiles = tile_split(G);
        Carver cv;
        uint64_t o_mask, o_offs, o_total;
        cv.add(&o_mask, 8 * G);
        cv.add(&o_offs, 8 * G);
        cv.add(&o_total, 8);
        Temp t(c);
        Staged sg;
        uint64_t xd, scr;
        settle(c, false);
        if (int st = stage(c, job, is_small(job), t, {}, cv.total, sg, xd, scr)) return st;
        uint64_t *d_mask = (uint64_t *)(scr + o_mask), *d_offs = (uint64_t *)(scr + o_offs);
        uint64_t *d_total = (uint64_t *)(scr + o_total);
        hipStream_t s = c->stream;
        int st = with_tables(sg, [&](const auto &tab) {
            return launch(c, "hash", [&] { return launch_tile(tab, G, kModeDiff, nullptr, d_mask, 0, s, tiles); });
        });
        if (st) return st;
        if ((st = launch(c, "classify", [&] { return launch_scan(d_mask, G, d_offs, d_total, SlotBump{}, s); })))
            return st;
        HIP_TRY(c, hipMemcpyAsync(&differing, d_total, 8, hipMemcpyDeviceToHost, s));
        HIP_TRY(c, hipStreamSynchronize(s));
    }
    if (h_differing) *h_differing = differing;
    if (h_distance) *h_distance = T ? (double)differing / (double)T : 0.0;
    return PCS_OK;
}

int pcs_bank_shrink(pcs_ctx *c, const pcs_bank_part *parts, uint32_t nparts, uint64_t n_entries,
                    const float *d_scores, uint64_t keep, uint32_t *d_kept)
{
    if (!c) return PCS_E_INVAL;
    if (nparts > 64) return fail(c, PCS_E_INVAL, "at most 64 bank parts");
    if (nparts && !parts) return fail(c, PCS_E_INVAL, "null parts");
    if (n_entries > UINT32_MAX) return fail(c, PCS_E_INVAL, "at most 2^32 - 1 bank entries (%llu given)",
                                            (unsigned long long)n_entries);
    if (keep > n_entries)
        return fail(c, PCS_E_INVAL, "keep %llu exceeds %llu entries", (unsigned long long)keep,
                    (unsigned long long)n_entries);
    if (n_entries && !d_scores) return fail(c, PCS_E_INVAL, "null scores");
    if ((uint64_t)d_scores & 3) return fail(c, PCS_E_INVAL, "scores must be 4-byte aligned");
    for (uint32_t p = 0; p < nparts; ++p) {
        const pcs_bank_part &q = parts[p];
        if (q.entry_bytes == 0) return fail(c, PCS_E_INVAL, "part %u: entry_bytes must be > 0", p);
        if (n_entries == 0) continue;
        if (!q.src || !q.dst) return fail(c, PCS_E_INVAL, "part %u: null address", p);
        if (q.entry_bytes > UINT64_MAX / n_entries) return fail(c, PCS_E_INVAL, "part %u: bank too large", p);
        const uint64_t sb = n_entries * q.entry_bytes, db = keep * q.entry_bytes;
        if (q.src > UINT64_MAX - sb || q.dst > UINT64_MAX - db)
            return fail(c, PCS_E_INVAL, "part %u: address range wraps", p);
        if (q.dst != q.src && db && q.dst < q.src + sb && q.src < q.dst + db)
            return fail(c, PCS_E_INVAL, "part %u: destination overlaps the source bank", p);
    }
    // The parts move in the same launches, so no part may write where another
    // part reads or writes.
    const auto overlap = [](uint64_t a, uint64_t na, uint64_t b, uint64_t nb) {
        return na && nb && a < b + nb && b < a + na;
    };
    for (uint32_t p = 0; p < nparts && n_entries; ++p)
        for (uint32_t q = 0; q < nparts; ++q) {
            if (p == q) continue;
            const pcs_bank_part &a = parts[p], &b = parts[q];
            if (overlap(a.dst, keep * a.entry_bytes, b.src, n_entries * b.entry_bytes) ||
                overlap(a.dst, keep * a.entry_bytes, b.dst, keep * b.entry_bytes))
                return fail(c, PCS_E_INVAL, "part %u: destination overlaps part %u", p, q);
        }
    if (n_entries == 0 || keep == 0) return PCS_OK;
    // Scratch: the kept indices (when the caller takes none), the state of a
    // large bank's selection, and, per in-place part, a staging area of keep
    // entries (slot j holds the source of destination j when that source is
    // itself a destination).  Keeping every entry leaves an in-place part as
    // it is: it moves nothing.
    const auto moves = [&](const pcs_bank_part &q) { return q.dst != q.src || keep < n_entries; };
    Temp t(c);
    Carver cv;
    uint64_t o_kept = 0, o_sel = 0;
    std::vector<uint64_t> o_stage(nparts, 0);
    if (!d_kept) cv.add(&o_kept, 4 * keep);
    const uint64_t sel_bytes = select_scratch_bytes((uint32_t)n_entries);
    if (sel_bytes) cv.add(&o_sel, sel_bytes);
    for (uint32_t p = 0; p < nparts; ++p)
        if (parts[p].dst == parts[p].src && moves(parts[p])) cv.add(&o_stage[p], keep * parts[p].entry_bytes);
    uint64_t base = 0;
    if (cv.total) {
        if (int e = temp_alloc(c, t, cv.total)) return e;
        base = c->arena_dev + t.off;
    }
    uint32_t *kept = d_kept ? d_kept : (uint32_t *)(base + o_kept);
    ShrinkParts P{};
    P.n = nparts;
    bool any_in_place = false;
    for (uint32_t p = 0; p < nparts; ++p) {
        const pcs_bank_part &q = parts[p];
        ShrinkPart &sp = P.p[p];
        sp.src = q.src;
        sp.dst = q.dst;
        sp.stage = q.dst == q.src && moves(q) ? base + o_stage[p] : 0;
        sp.eb = q.entry_bytes;
        const auto aligned = [&](uint64_t g) {
            return q.entry_bytes % g == 0 && q.src % g == 0 && q.dst % g == 0 && sp.stage % g == 0;
        };
        sp.g = aligned(16) ? 16 : aligned(4) ? 4 : 1;
        sp.spe = (q.entry_bytes / sp.g + 255) / 256;
        sp.item_begin = P.items;
        if (moves(q)) P.items += keep * sp.spe;  // else the part has no items
        any_in_place = any_in_place || sp.stage != 0;
    }
    for (uint32_t step = 0; step < select_steps((uint32_t)n_entries); ++step)
        if (int st = launch(c, "shrink", [&] {
                return launch_shrink_select(d_scores, (uint32_t)n_entries, (uint32_t)keep, kept,
                                            sel_bytes ? base + o_sel : 0, step, c->stream);
            }))
            return st;
    if (P.items == 0) return PCS_OK;  // no part moves (none given, or in place keeping every entry)
    if (any_in_place)
        if (int st = launch(c, "shrink", [&] { return launch_move_entries(P, kept, keep, true, c->stream); }))
            return st;
    return launch(c, "shrink", [&] { return launch_move_entries(P, kept, keep, false, c->stream); });
}

int pcs_checkpoint(pcs_ctx *c, const pcs_buf *plan, uint32_t n, pcs_snap parent, uint32_t flags,
                   uint64_t *d_hashes, uint64_t *d_roots, uint64_t *d_sroot, pcs_snap *out)
{
    if (!c) return PCS_E_INVAL;
    if (!out) return fail(c, PCS_E_INVAL, "null output handle");
    if (n && !plan) return fail(c, PCS_E_INVAL, "null plan");
    if (flags & ~PCS_CKPT_HASH) return fail(c, PCS_E_INVAL, "unknown flags");
    if (parent == 0) {
        const uint32_t nb[1] = {n};
        return checkpoint_full(c, plan, nb, 1, flags, d_hashes, d_roots, d_sroot, out);
    }

    // Incremental checkpoint against `parent`.
    auto par = lookup(c, parent);
    if (!par) return fail(c, PCS_E_HANDLE, "unknown parent handle %llu", (unsigned long long)parent);
    if (!par->has_hashes) return fail(c, PCS_E_INVAL, "parent snapshot holds no fingerprints");
    if (par->nbufs != n) return fail(c, PCS_E_INVAL, "plan has %u buffers, parent %u", n, par->nbufs);
    Job job;
    if (int st = add_buffers(c, job, plan, n, 0)) return st;
    const uint64_t T = job.nchunks, G = job.ngroups;

    // Metadata block [hashes 8T][manifest 8T][roots 8(n+1)] from the bottom.
    // The stored chunks go to slots the device places in a segment (see
    // Segment): the host claims the worst case (one slot per chunk) until the
    // stream has produced the count.  When no segment can hold the worst case
    // even after every pending call has settled, the call takes the exact
    // path: it waits for its own count, then allocates exactly that many slots.
    const uint64_t hashes_rel = 0, manifest_rel = 8 * T, roots_rel = 16 * T;
    const uint64_t meta = roots_rel + 8 * (n + 1);
    if (c->free_pairs.empty()) settle(c, true);
    if (c->free_pairs.empty()) return fail(c, PCS_E_NOMEM, "too many incremental snapshots in flight");
    uint64_t boff;
    if (!alloc_block(c, meta, &boff))
        return fail(c, PCS_E_NOMEM, "arena cannot hold incremental snapshot metadata (%llu bytes)",
                    (unsigned long long)meta);
    auto node = std::make_shared<SnapNode>();
    node->ctx = c;
    node->block_off = boff;
    node->block_bytes = meta;
    node->nbufs = n;
    node->incremental = true;
    node->has_hashes = true;
    for (uint32_t b = 0; b < n; ++b) {
        node->bufs.push_back(job.lays[b]);
        node->chunk_begin.push_back(job.bufs[b].chunk_begin);
        node->state_bytes += job.lays[b].nbytes;
    }
    node->total_chunks = T;
    node->hashes_off = boff + hashes_rel;
    node->manifest_off = boff + manifest_rel;
    node->roots_off = boff + roots_rel;
    node->parent = par;
    const uint64_t worst = T * kChunk;
    std::shared_ptr<Segment> seg = T ? segment_for(c, worst) : nullptr;
    const bool exact = T && !seg;

    // A small job fingerprints and diffs as sub-tiles; the Merkle lists then
    // reduce one node per sub-tile (an aligned 8-chunk subtree).
    const uint32_t tiles = tile_split(G);
    const uint64_t per_tile = kGroupChunks / tiles;
    std::vector<MerkleList> lists;
    for (uint32_t b = 0; b < n; ++b) {
        JobBuf &jb = job.bufs[b];
        jb.hash_dst[0] = c->arena_dev + node->hashes_off + 8 * jb.chunk_begin;
        jb.hash_dst[1] = d_hashes ? (uint64_t)(d_hashes + jb.chunk_begin) : 0;
        jb.manifest = c->arena_dev + node->manifest_off + 8 * jb.chunk_begin;
        jb.parent_hash = c->arena_dev + par->hashes_off + 8 * par->chunk_begin[b];
        jb.parent_chunks = par->bufs[b].nchunks;
        if (par->incremental) {
            jb.parent_manifest = c->arena_dev + par->manifest_off + 8 * par->chunk_begin[b];
        } else {
            jb.parent_slot0 = par->payload_off + par->comp_off[b];
        }
        lists.push_back({jb.group_begin * tiles, div_up(jb.nchunks, per_tile),
                         {c->arena_dev + node->roots_off + 8 * b, d_roots ? (uint64_t)(d_roots + b) : 0}});
    }
    lists.push_back({0, n, {c->arena_dev + node->roots_off + 8 * n, (uint64_t)d_sroot}});

    // Where the scan places the slots: in the segment (pipelined), nowhere
    // (exact: the host places them once it has read the count from pair 0),
    // or no slots at all (no chunks).
    uint32_t pair = 0;
    SlotBump bump{nullptr, nullptr, 0, nullptr, nullptr};
    if (seg) {
        pair = c->free_pairs.back();
        c->free_pairs.pop_back();
        uint64_t *words = (uint64_t *)c->bump_dev;
        bump = SlotBump{words + 2 * c->bump_par, words + 2 * (c->bump_par ^ 1), seg->started ? 0 : seg->hi,
                        (uint64_t *)c->top_dev, &c->counts_dev[2 * pair]};
        c->bump_par ^= 1;
        seg->started = true;
        seg->claim += worst;
        ++seg->pending;
    } else if (exact) {
        bump.host = &c->counts_dev[0];
    }
    // On an error before the call is recorded as pending, its claim goes back
    // and the segment closes: a scan this call had already enqueued moves the
    // device's bump word below the slots the host counts, so no later call
    // may be placed after it in this segment (a new segment resets the word).
    bool recorded = !seg;
    struct Undo {
        pcs_ctx *c;
        std::shared_ptr<Segment> &seg;
        uint64_t worst;
        uint32_t pair;
        bool &recorded;
        ~Undo()
        {
            if (recorded) return;
            seg->claim -= worst;
            --seg->pending;
            seg->open = false;
            if (c->seg == seg) c->seg.reset();
            c->free_pairs.push_back(pair);
            retire_if_idle(c, seg);
        }
    } undo{c, seg, worst, pair, recorded};

    // A small job (tables in kernel arguments) on the pipelined path runs as
    // two launches: fingerprint+diff, then the Merkle lists, the scan, the
    // slot placement and the dirty copy.
    const bool small = is_small(job) && !exact && G <= kScanCompactMaxGroups;
    Carver cv;
    uint64_t o_nodes, o_sa, o_sb, o_roots, o_mask, o_offs, o_total;
    cv.add(&o_nodes, 8 * G * tiles);
    cv.add(&o_sa, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_sb, 8 * std::max<uint64_t>(G * tiles, n));
    cv.add(&o_roots, 8 * n);
    cv.add(&o_mask, 8 * G);
    cv.add(&o_offs, 8 * G);
    cv.add(&o_total, 8);
    Temp t(c);
    Staged sg;
    uint64_t lists_dev, scr;
    if (int st = stage(c, job, small, t, small ? std::vector<uint8_t>() : bytes_of(lists), cv.total, sg, lists_dev, scr))
        return st;
    uint64_t *d_nodes = (uint64_t *)(scr + o_nodes);
    uint64_t *d_sa = (uint64_t *)(scr + o_sa), *d_sb = (uint64_t *)(scr + o_sb);
    uint64_t *d_roots_tmp = (uint64_t *)(scr + o_roots);
    uint64_t *d_mask = (uint64_t *)(scr + o_mask), *d_offs = (uint64_t *)(scr + o_offs);
    uint64_t *d_total = (uint64_t *)(scr + o_total);
    const uint64_t *top_word = (const uint64_t *)c->top_dev;
    hipStream_t s = c->stream;
    int st = with_tables(sg, [&](const auto &tab) {
        return launch(c, "incremental", [&] {
            return launch_tile(tab, G, kModeDiff, d_nodes, d_mask, 0, s, tiles);
        });
    });
    if (st) return st;
    if (small) {
        const ArgLists al = arg_lists(lists, n);
        if ((st = launch(c, "incremental", [&] {
                 return launch_merkle_scan_place(al, d_nodes, d_sa, d_sb, sg.arg, G, d_mask, bump, d_total,
                                                 c->arena_dev, s);
             })))
            return st;
    } else {
        if ((st = run_merkle(c, small, lists, n, lists_dev, d_nodes, d_sa, d_sb, d_roots_tmp))) return st;
        if ((st = launch(c, "incremental", [&] { return launch_scan(d_mask, G, d_offs, d_total, bump, s); })))
            return st;
        if (exact) {
            HIP_TRY(c, hipEventRecord(c->exact_ev, s));
            HIP_TRY(c, hipEventSynchronize(c->exact_ev));
            const uint64_t dirty = c->counts[0];
            uint64_t poff = 0;
            if (dirty && !alloc_block_top(c, dirty * kChunk, &poff))
                return fail(c, PCS_E_NOMEM, "arena cannot hold %llu stored chunks of an incremental snapshot "
                            "(its fingerprint outputs were written)", (unsigned long long)dirty);
            node->pay_off = node->payload_off = poff;
            node->pay_bytes = node->payload_bytes = dirty * kChunk;
            node->pay_top = poff + dirty * kChunk;
            c->counts[1] = node->pay_top;
            HIP_TRY(c, hipMemcpyAsync((void *)c->top_dev, &c->counts[1], 8, hipMemcpyHostToDevice, s));
        }
        st = with_tables(sg, [&](const auto &tab) {
            return launch(c, "incremental", [&] {
                return launch_place_dirty(tab, G, d_mask, d_offs, top_word, c->arena_dev, s);
            });
        });
        if (st) return st;
    }
    if (seg) {
        PendingCall pc;
        pc.node = node;
        pc.seg = seg;
        pc.worst = worst;
        pc.pair = pair;
        HIP_TRY(c, hipEventCreateWithFlags(&pc.ev, hipEventDisableTiming));
        const hipError_t e = hipEventRecord(pc.ev, s);
        if (e != hipSuccess) {
            (void)hipEventDestroy(pc.ev);
            return hip_fail(c, e, "hipEventRecord");
        }
        node->settled = false;
        c->pending.push_back(pc);
        recorded = true;
    }
    *out = new_handle(c, node);
    return PCS_OK;
}

int pcs_checkpoint_batch(pcs_ctx *c, const pcs_buf *plans, const uint32_t *nbufs, uint32_t sessions, uint32_t flags,
                         uint64_t *d_hashes, uint64_t *d_roots, uint64_t *d_sroots, pcs_snap *out)
{
    if (!c) return PCS_E_INVAL;
    if (sessions && (!nbufs || !out)) return fail(c, PCS_E_INVAL, "null argument");
    if (flags & ~PCS_CKPT_HASH) return fail(c, PCS_E_INVAL, "unknown flags");
    uint64_t nb = 0;
    for (uint32_t s = 0; s < sessions; ++s) nb += nbufs[s];
    if (nb && !plans) return fail(c, PCS_E_INVAL, "null plans");
    return checkpoint_full(c, plans, nbufs, sessions, flags, d_hashes, d_roots, d_sroots, out);
}

int pcs_restore_batch(pcs_ctx *c, const pcs_snap *snaps, uint32_t m, const pcs_buf *dsts, const uint32_t *nbufs)
{
    return restore_impl(c, snaps, m, dsts, nbufs, true);
}

int pcs_restore_verify(pcs_ctx *c, pcs_snap snap, const pcs_buf *dst, uint32_t n, uint64_t *d_bad_bitmap,
                       uint8_t *d_bad_labels)
{
    if (!c) return PCS_E_INVAL;
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->has_hashes) return fail(c, PCS_E_INVAL, "snapshot holds no fingerprints to verify against");
    if (n != nd->nbufs) return fail(c, PCS_E_SHAPE, "snapshot holds %u buffers, %u destinations given", nd->nbufs, n);
    if (n && !dst) return fail(c, PCS_E_INVAL, "null destinations");
    Job job;
    if (int st = add_buffers(c, job, dst, n, 0)) return st;
    if (job.ngroups && !d_bad_bitmap) return fail(c, PCS_E_INVAL, "null mismatch bitmap");
    for (uint32_t k = 0; k < n; ++k) {
        const Layout &want = nd->bufs[k], &got = job.lays[k];
        if (want.kind != got.kind || want.nbytes != got.nbytes ||
            (want.kind == PCS_RING && (want.row_bytes != got.row_bytes || want.window != got.window ||
                                       want.outer != got.outer)))
            return fail(c, PCS_E_SHAPE, "buffer %u: destination layout differs from the snapshot", k);
        JobBuf &jb = job.bufs[k];
        if (nd->incremental)
            jb.manifest = c->arena_dev + nd->manifest_off + 8 * nd->chunk_begin[k];
        else
            jb.payload = c->arena_dev + nd->payload_off + nd->comp_off[k];
        jb.parent_hash = c->arena_dev + nd->hashes_off + 8 * nd->chunk_begin[k];
    }
    if (n == 0) return PCS_OK;
    Temp t(c);
    Staged sg;
    uint64_t xd, scr;
    if (int st = stage(c, job, is_small(job), t, {}, 0, sg, xd, scr)) return st;
    const uint64_t G = job.ngroups;
    return with_tables(sg, [&](const auto &tab) {
        if (int st = launch(c, "verify", [&] {
                return launch_tile(tab, G, kModeVerify, nullptr, d_bad_bitmap, c->arena_dev, c->stream, 1, c->dev);
            }))
            return st;
        if (!d_bad_labels) return (int)PCS_OK;
        return launch(c, "verify", [&] { return launch_labels(tab, d_bad_bitmap, d_bad_labels, c->stream); });
    });
}

int pcs_snapshot_view(pcs_ctx *c, pcs_snap snap, uint64_t *d_payload, uint64_t *bytes)
{
    if (!c) return PCS_E_INVAL;
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->settled) settle(c, true);
    if (d_payload) *d_payload = c->arena_dev + nd->payload_off;
    if (bytes) *bytes = nd->payload_bytes;
    return PCS_OK;
}

int pcs_restore(pcs_ctx *c, pcs_snap snap, const pcs_buf *dst, uint32_t n)
{
    return pcs_restore_batch(c, &snap, 1, dst, &n);
}

int pcs_fork(pcs_ctx *c, pcs_snap snap, pcs_snap *out)
{
    if (!c) return PCS_E_INVAL;
    if (!out) return fail(c, PCS_E_INVAL, "null output handle");
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    *out = new_handle(c, nd);
    return PCS_OK;
}

int pcs_delete(pcs_ctx *c, pcs_snap snap)
{
    if (!c) return PCS_E_INVAL;
    auto it = c->handles.find(snap);
    if (it == c->handles.end()) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    c->handles.erase(it);
    return PCS_OK;
}

int pcs_snapshot_info(pcs_ctx *c, pcs_snap snap, pcs_snap_info *out)
{
    if (!c) return PCS_E_INVAL;
    if (!out) return fail(c, PCS_E_INVAL, "null output");
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->settled) settle(c, true);
    memset(out, 0, sizeof *out);
    out->state_bytes = nd->state_bytes;
    out->stored_bytes = nd->payload_bytes;
    out->total_chunks = nd->total_chunks;
    out->dirty_chunks = nd->incremental ? nd->payload_bytes / kChunk : nd->total_chunks;
    out->nbufs = nd->nbufs;
    out->incremental = nd->incremental;
    out->has_hashes = nd->has_hashes;
    return PCS_OK;
}

int pcs_snapshot_payload(pcs_ctx *c, pcs_snap snap, void *d_dst, uint64_t cap)
{
    if (!c) return PCS_E_INVAL;
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->settled) settle(c, true);
    if (cap < nd->payload_bytes) return fail(c, PCS_E_INVAL, "destination holds %llu bytes, payload is %llu",
                                             (unsigned long long)cap, (unsigned long long)nd->payload_bytes);
    if (nd->payload_bytes == 0) return PCS_OK;
    if (!d_dst) return fail(c, PCS_E_INVAL, "null destination");
    if (nd->incremental) {
        // Stored slots grow downwards from the top of the reservation; hand
        // them out in increasing slot order.
        if ((uint64_t)d_dst % 16) return fail(c, PCS_E_INVAL, "destination must be 16-byte aligned");
        return launch(c, "copy", [&] {
            return launch_reverse_slots(c->arena_dev + nd->pay_top, (uint64_t)d_dst, nd->payload_bytes / kChunk,
                                        c->stream);
        });
    }
    HIP_TRY(c, hipMemcpyAsync(d_dst, (void *)(c->arena_dev + nd->payload_off), nd->payload_bytes,
                              hipMemcpyDeviceToDevice, c->stream));
    return PCS_OK;
}

int pcs_snapshot_hashes(pcs_ctx *c, pcs_snap snap, uint64_t *d_dst, uint64_t cap)
{
    if (!c) return PCS_E_INVAL;
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->has_hashes) return fail(c, PCS_E_INVAL, "snapshot holds no fingerprints");
    if (cap < nd->total_chunks) return fail(c, PCS_E_INVAL, "destination too small");
    if (nd->total_chunks == 0) return PCS_OK;
    if (!d_dst) return fail(c, PCS_E_INVAL, "null destination");
    HIP_TRY(c, hipMemcpyAsync(d_dst, (void *)(c->arena_dev + nd->hashes_off), 8 * nd->total_chunks,
                              hipMemcpyDeviceToDevice, c->stream));
    return PCS_OK;
}

int pcs_arena_stats(pcs_ctx *c, uint64_t *used, uint64_t *free_bytes, uint64_t *largest, uint64_t *live)
{
    if (!c) return PCS_E_INVAL;
    settle(c, false);
    // Not counted as used: the library's own unit, and the part of every
    // live segment that neither a snapshot's slots nor a pending call's
    // worst case claims.
    uint64_t idle = 0;
    std::vector<const Segment *> seen;
    auto count = [&](const Segment *g) {
        if (!g || g->retired || std::find(seen.begin(), seen.end(), g) != seen.end()) return;
        seen.push_back(g);
        idle += (g->hi - g->lo) - g->claim;
    };
    count(c->seg.get());
    for (const auto &p : c->pending) count(p.seg.get());
    const uint64_t in_use = c->arena.used() - kAlign - idle;
    if (used) *used = in_use;
    if (free_bytes) *free_bytes = c->arena.size() - kAlign - in_use;
    if (largest) *largest = c->arena.largest();
    if (live) *live = c->handles.size();
    return PCS_OK;
}

int pcs_set_timing(pcs_ctx *c, int mode)
{
    if (!c) return PCS_E_INVAL;
    if (mode != PCS_TIMING_OFF && mode != PCS_TIMING_EVENTS && mode != PCS_TIMING_DISPATCH)
        return fail(c, PCS_E_INVAL, "timing mode %d: 0, 1 or 2", mode);
    c->timing = mode;
    return PCS_OK;
}

int pcs_kernel_time(pcs_ctx *c, const char *name, uint64_t *launches, double *total_ms)
{
    if (!c || !name) return PCS_E_INVAL;
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    double ms = 0;
    uint64_t k = 0;
    hipError_t e = hipSuccess;
    auto it = c->timers.find(name);
    if (it != c->timers.end()) {
        // Every pair is destroyed and the name's record cleared, also when a
        // query fails (then the first failure is returned).
        for (auto &ab : it->second) {
            float t = 0;
            const hipError_t q = e == hipSuccess ? hipEventElapsedTime(&t, ab.first, ab.second) : e;
            if (q == hipSuccess) {
                ms += t;
                ++k;
            } else {
                e = q;
            }
            (void)hipEventDestroy(ab.first);
            (void)hipEventDestroy(ab.second);
        }
        c->timers.erase(it);
    }
    if (e != hipSuccess) return hip_fail(c, e, "hipEventElapsedTime");
    if (launches) *launches = k;
    if (total_ms) *total_ms = ms;
    return PCS_OK;
}

int pcs_export(pcs_ctx *c, pcs_snap snap, void *h_dst, uint64_t cap, uint64_t *written)
{
    if (!c) return PCS_E_INVAL;
    auto nd = lookup(c, snap);
    if (!nd) return fail(c, PCS_E_HANDLE, "unknown handle %llu", (unsigned long long)snap);
    if (!nd->settled) settle(c, true);
    const uint32_t n = nd->nbufs;
    const uint64_t T = nd->total_chunks;
    ImageLayout L;
    if (!image_layout(nd->bufs, T, &L)) return fail(c, PCS_E_INVAL, "snapshot too large for an image");
    if (written) *written = L.size;
    if (!h_dst) return PCS_OK;
    if (cap < L.size) return fail(c, PCS_E_INVAL, "image needs %llu bytes", (unsigned long long)L.size);
    uint8_t *img = (uint8_t *)h_dst;
    write_image_header(img, nd->bufs, T, nd->state_bytes, L);
    hipStream_t s = c->stream;
    // Canonical payload: a full snapshot already is one; an incremental one is
    // laid out flat through its manifest into scratch first.
    Temp t(c);
    uint64_t payload_dev = c->arena_dev + nd->payload_off;
    if (nd->incremental && L.payload) {
        if (int st = temp_alloc(c, t, L.payload)) return st;
        payload_dev = c->arena_dev + t.off;
        HIP_TRY(c, hipMemsetAsync((void *)payload_dev, 0, L.payload, s));
        std::vector<pcs_buf> flat(n);
        for (uint32_t b = 0; b < n; ++b) {
            memset(&flat[b], 0, sizeof(pcs_buf));
            flat[b].ptr = payload_dev + L.comp_off[b];
            flat[b].nbytes = nd->bufs[b].nbytes;
            flat[b].kind = PCS_FLAT;
        }
        if (int st = restore_impl(c, &snap, 1, flat.data(), &n, false)) return st;
    }
    // Fingerprints: stored ones, or computed from the payload.
    Temp th(c);
    uint64_t hashes_dev = c->arena_dev + nd->hashes_off, roots_dev = c->arena_dev + nd->roots_off;
    if (!nd->has_hashes) {
        if (int st = temp_alloc(c, th, 8 * T + 8 * (n + 1))) return st;
        hashes_dev = c->arena_dev + th.off;
        roots_dev = hashes_dev + 8 * T;
        std::vector<uint64_t> addr(n), nb(n);
        for (uint32_t b = 0; b < n; ++b) {
            addr[b] = payload_dev + L.comp_off[b];
            nb[b] = nd->bufs[b].nbytes;
        }
        if (int st = fingerprint_regions(c, addr, nb, (uint64_t *)hashes_dev, (uint64_t *)roots_dev,
                                         (uint64_t *)(roots_dev + 8 * n)))
            return st;
    }
    // The copies write into the caller's image: an error after the first one
    // was enqueued waits for the stream before returning, so no copy is still
    // in flight when the caller regains the image.
    hipError_t e = hipMemcpyAsync(img + L.roots_off, (void *)roots_dev, 8 * (n + 1), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && T) e = hipMemcpyAsync(img + L.hashes_off, (void *)hashes_dev, 8 * T, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && L.payload)
        e = hipMemcpyAsync(img + L.data_off, (void *)payload_dev, L.payload, hipMemcpyDeviceToHost, s);
    const hipError_t w = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(c, e, "image download");
    if (w != hipSuccess) return hip_fail(c, w, "hipStreamSynchronize");
    return PCS_OK;
}

int pcs_import(pcs_ctx *c, const void *h_src, uint64_t size, pcs_snap *out)
{
    if (!c) return PCS_E_INVAL;
    if (!out || !h_src) return fail(c, PCS_E_INVAL, "null argument");
    const uint8_t *img = (const uint8_t *)h_src;
    std::vector<Layout> lays;
    ImageLayout L;
    std::string why;
    if (int st = parse_image_header(img, size, &lays, &L, &why)) return fail(c, st, "%s", why.c_str());
    const uint32_t n = (uint32_t)lays.size();
    const uint64_t T = get64(img + 16), payload = L.payload;

    // A full snapshot with fingerprints, filled from the image.
    Job job;
    job.lays = lays;
    uint64_t cb = 0;
    for (auto &y : lays) {
        JobBuf jb{};
        jb.nbytes = y.nbytes;
        jb.nchunks = y.nchunks;
        jb.chunk_begin = cb;
        cb += y.nchunks;
        job.bufs.push_back(jb);
    }
    const FullPlan fp = full_plan(job, 0, n, T, true);
    uint64_t boff;
    if (!alloc_block(c, fp.block, &boff))
        return fail(c, PCS_E_NOMEM, "arena cannot hold the imported snapshot (%llu bytes)", (unsigned long long)fp.block);
    auto node = make_node(c, job, 0, n, fp, boff, true);
    // Scratch for the verification, reserved before anything reads the
    // caller's image, so that no error return leaves a copy from it in flight.
    Temp t(c);
    if (int st = temp_alloc(c, t, 8 * T + 8 * (n + 1))) return st;
    const uint64_t h_dev = c->arena_dev + t.off, r_dev = h_dev + 8 * T;
    hipStream_t s = c->stream;
    // Any failure from here on first waits for the copies already enqueued.
    auto drain = [&](int st) {
        (void)hipStreamSynchronize(s);
        return st;
    };
    hipError_t e = hipMemcpyAsync((void *)(c->arena_dev + node->roots_off), img + L.roots_off, 8 * (n + 1),
                                  hipMemcpyHostToDevice, s);
    if (e == hipSuccess && T)
        e = hipMemcpyAsync((void *)(c->arena_dev + node->hashes_off), img + L.hashes_off, 8 * T,
                           hipMemcpyHostToDevice, s);
    if (e == hipSuccess && payload)
        e = hipMemcpyAsync((void *)(c->arena_dev + node->payload_off), img + L.data_off, payload,
                           hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return drain(hip_fail(c, e, "image upload"));
    // Verify: fingerprint the imported payload and compare with the image.
    std::vector<uint64_t> addr(n), nb(n);
    for (uint32_t b = 0; b < n; ++b) {
        addr[b] = c->arena_dev + node->payload_off + node->comp_off[b];
        nb[b] = lays[b].nbytes;
    }
    if (int st = fingerprint_regions(c, addr, nb, (uint64_t *)h_dev, (uint64_t *)r_dev, (uint64_t *)(r_dev + 8 * n)))
        return drain(st);
    std::vector<uint64_t> got(T + n + 1);
    e = hipMemcpyAsync(got.data(), (void *)h_dev, 8 * (T + n + 1), hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return drain(hip_fail(c, e, "fingerprint download"));
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return drain(hip_fail(c, e, "hipStreamSynchronize"));
    for (uint64_t i = 0; i < T; ++i)
        if (got[i] != get64(img + L.hashes_off + 8 * i))
            return fail(c, PCS_E_CORRUPT, "chunk %llu does not match its fingerprint", (unsigned long long)i);
    for (uint32_t b = 0; b <= n; ++b)
        if (got[T + b] != get64(img + L.roots_off + 8 * b))
            return fail(c, PCS_E_CORRUPT, "root %u does not match", b);
    *out = new_handle(c, node);
    return PCS_OK;
}

int pcs_discover(pcs_ctx *c, const pcs_buf *comps, uint32_t k, double eps, int32_t control, pcs_probe_fn probe,
                 void *user, pcs_discovery *out)
{
    if (!c) return PCS_E_INVAL;
    if (!out) return fail(c, PCS_E_INVAL, "null result");
    if (!probe) return fail(c, PCS_E_INVAL, "null probe");
    if (k > PCS_DISCOVER_MAX) return fail(c, PCS_E_INVAL, "at most %u components", PCS_DISCOVER_MAX);
    if (k && !comps) return fail(c, PCS_E_INVAL, "null components");
    if (!(eps >= 0)) return fail(c, PCS_E_INVAL, "eps must be a number >= 0");
    if (control >= (int32_t)k) return fail(c, PCS_E_INVAL, "control component %d out of range", control);
    std::vector<uint64_t> chunks(k ? k : 1);
    if (k) {
        if (int st = pcs_chunk_counts(comps, k, chunks.data(), nullptr))
            return fail(c, st, "invalid component descriptor");
    }
    if (control >= 0 && chunks[control] == 0)
        return fail(c, PCS_E_INVAL, "control component %d is empty", control);
    memset(out, 0, sizeof *out);
    out->d_control = -1;
    out->control_ok = -1;
    uint32_t probes = 0;

    // One probe: a full snapshot of the masked components (with component
    // `corrupt` given a wrong value), the caller's probe, then the delete.
    auto run = [&](const uint8_t *mask, int32_t corrupt, double *d) -> int {
        std::vector<pcs_buf> plan;
        int32_t pos = -1;
        for (uint32_t i = 0; i < k; ++i) {
            if (!mask[i]) continue;
            if ((int32_t)i == corrupt) pos = (int32_t)plan.size();
            plan.push_back(comps[i]);
        }
        pcs_snap snap = 0;
        if (int st = pcs_checkpoint(c, plan.data(), (uint32_t)plan.size(), 0, 0, nullptr, nullptr, nullptr, &snap))
            return st;
        if (pos >= 0) {
            const auto nd = lookup(c, snap);
            const uint64_t addr = c->arena_dev + nd->payload_off + nd->comp_off[pos];
            if (int st = launch(c, "flip", [&] { return launch_flip_bit(addr, c->stream); })) {
                pcs_delete(c, snap);
                return st;
            }
        }
        ++probes;
        double dv = 0;
        const int r = probe(user, snap, mask, k, &dv);
        pcs_delete(c, snap);
        if (r != 0) return fail(c, PCS_E_PROBE, "probe returned %d", r);
        if (!(dv >= 0)) return fail(c, PCS_E_PROBE, "probe returned a negative or NaN distance");
        *d = dv;
        return PCS_OK;
    };

    uint8_t mask[PCS_DISCOVER_MAX], cur[PCS_DISCOVER_MAX];
    // 1. necessity: leave each component out in turn.
    for (uint32_t i = 0; i < k; ++i) {
        memset(mask, 1, k);
        mask[i] = 0;
        double d = 0;
        if (int st = run(mask, -1, &d)) return st;
        out->d_without[i] = d;
        out->necessary[i] = d > eps ? 1 : 0;
    }
    // 2. sufficiency: exactly the necessary set.
    uint32_t in = 0;
    for (uint32_t i = 0; i < k; ++i) {
        cur[i] = out->necessary[i];
        in += cur[i];
    }
    double d = 0;
    if (int st = run(cur, -1, &d)) return st;
    out->d_necessary = d;
    // 3. redundancy fallback: add the component that most reduces D.
    while (d > eps && in < k) {
        int32_t best = -1;
        double best_d = 0;
        for (uint32_t j = 0; j < k; ++j) {
            if (cur[j]) continue;
            memcpy(mask, cur, k);
            mask[j] = 1;
            double dj = 0;
            if (int st = run(mask, -1, &dj)) return st;
            if (best < 0 || dj < best_d) {
                best = (int32_t)j;
                best_d = dj;
            }
        }
        cur[best] = 1;
        ++in;
        out->added[out->n_added++] = (uint32_t)best;
        d = best_d;
    }
    memcpy(out->pcs, cur, k);
    out->d_final = d;
    out->converged = d <= eps ? 1 : 0;
    // The control: the full state with one component given a wrong value.
    if (control >= 0) {
        memset(mask, 1, k);
        double dc = 0;
        if (int st = run(mask, control, &dc)) return st;
        out->d_control = dc;
        out->control_ok = dc > eps ? 1 : 0;
    }
    out->probes = probes;
    return PCS_OK;
}

}  // extern "C"

// Host-only tests of libpcs's runtime logic (no GPU involved):
//   - the arena sub-allocator against a brute-force occupancy model;
//   - plan descriptors (flat buffers, ring windows) against the ring's
//     defining index map, logical row t of ring o at physical row
//     (head + t) mod capacity, and the validation of bad descriptors;
//   - the XCD tile order of the tile kernels (a partition of the job's
//     tiles, and the one-tile-per-workgroup order written out);
//   - the snapshot image header: round trips, every single-field
//     corruption, a crafted size that wraps 64-bit arithmetic, random
//     mutations and truncations (an accepted header must name only regions
//     inside the image).
// Built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_logic.py; prints "ok" and exits 0 when every check holds.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>
#include <vector>

#include "../../paper_2607_21686_amd/csrc/pcs_host.h"

using namespace pcs;

static int g_checks = 0;
#define CHECK(cond)                                                                     \
    do {                                                                                \
        ++g_checks;                                                                     \
        if (!(cond)) {                                                                  \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond);  \
            exit(1);                                                                    \
        }                                                                               \
    } while (0)

// ------------------------------------------------------------------ arena

// Occupancy model: one flag per 4096-byte unit.
struct Model {
    std::vector<uint8_t> used;
    explicit Model(uint64_t units) : used(units, 0) {}
    // Maximal free runs (start unit, length in units), in address order.
    std::vector<std::pair<uint64_t, uint64_t>> free_runs() const
    {
        std::vector<std::pair<uint64_t, uint64_t>> r;
        for (uint64_t i = 0; i < used.size();) {
            if (used[i]) {
                ++i;
                continue;
            }
            uint64_t j = i;
            while (j < used.size() && !used[j]) ++j;
            r.push_back({i, j - i});
            i = j;
        }
        return r;
    }
};

static uint64_t units_of(uint64_t bytes) { return bytes == 0 ? 1 : (bytes + kAlign - 1) / kAlign; }

static void check_arena_matches(const Arena &a, const Model &m)
{
    const auto runs = m.free_runs();
    const auto &fr = a.free_ranges();
    CHECK(fr.size() == runs.size());  // the free map stays coalesced
    size_t k = 0;
    uint64_t largest = 0, free_units = 0;
    for (auto &kv : fr) {
        CHECK(kv.first == runs[k].first * kAlign);
        CHECK(kv.second == runs[k].second * kAlign);
        largest = std::max(largest, kv.second);
        free_units += runs[k].second;
        ++k;
    }
    CHECK(a.largest() == largest);
    CHECK(a.used() == (m.used.size() - free_units) * kAlign);
}

static void test_arena(uint64_t seed)
{
    std::mt19937_64 rng(seed);
    const uint64_t units = 1 + rng() % 600;
    Arena a;
    a.init(units * kAlign);
    Model m(units);
    struct Live {
        uint64_t off, bytes;
    };
    std::vector<Live> live;
    check_arena_matches(a, m);
    for (int op = 0; op < 3000; ++op) {
        const uint64_t r = rng() % 100;
        if (r < 55 || live.empty()) {
            // Request sizes: 0, exact units, and ragged byte counts.
            uint64_t bytes;
            switch (rng() % 4) {
            case 0: bytes = 0; break;
            case 1: bytes = (1 + rng() % 24) * kAlign; break;
            default: bytes = 1 + rng() % (24 * kAlign); break;
            }
            const uint64_t u = units_of(bytes);
            const bool top = rng() % 3 == 0;
            // Expected placement from the model: first fit (lowest run that
            // holds it, at its start) or top fit (highest such run, at its end).
            const auto runs = m.free_runs();
            int64_t want = -1;
            if (!top) {
                for (auto &fr : runs)
                    if (fr.second >= u) {
                        want = (int64_t)fr.first;
                        break;
                    }
            } else {
                for (auto it = runs.rbegin(); it != runs.rend(); ++it)
                    if (it->second >= u) {
                        want = (int64_t)(it->first + it->second - u);
                        break;
                    }
            }
            uint64_t off = ~0ULL;
            const bool ok = top ? a.alloc_top(bytes, &off) : a.alloc(bytes, &off);
            CHECK(ok == (want >= 0));
            if (ok) {
                CHECK(off % kAlign == 0);
                CHECK(off / kAlign == (uint64_t)want);
                CHECK(off / kAlign + u <= units);
                for (uint64_t i = 0; i < u; ++i) {
                    CHECK(!m.used[off / kAlign + i]);
                    m.used[off / kAlign + i] = 1;
                }
                live.push_back({off, bytes});
            }
        } else {
            const size_t i = rng() % live.size();
            const Live l = live[i];
            live[i] = live.back();
            live.pop_back();
            a.release(l.off, l.bytes);
            for (uint64_t k = 0; k < units_of(l.bytes); ++k) m.used[l.off / kAlign + k] = 0;
        }
        check_arena_matches(a, m);
    }
    for (auto &l : live) a.release(l.off, l.bytes);
    CHECK(a.used() == 0);
    CHECK(a.free_ranges().size() == 1 && a.largest() == units * kAlign);

    // Requests no arena can hold fail without touching the free map.
    uint64_t off;
    CHECK(!a.alloc(UINT64_MAX, &off));
    CHECK(!a.alloc_top(UINT64_MAX - 5, &off));
    CHECK(!a.alloc(units * kAlign + 1, &off));
    CHECK(a.used() == 0 && a.largest() == units * kAlign);
}

// ------------------------------------------------------------------ descriptors

static pcs_buf flat_buf(uint64_t ptr, uint64_t nbytes)
{
    pcs_buf b{};
    b.ptr = ptr;
    b.nbytes = nbytes;
    b.kind = PCS_FLAT;
    return b;
}

static pcs_buf ring_buf(uint64_t ptr, uint64_t outer, uint64_t cap, uint64_t row, uint64_t head, uint64_t window,
                        uint64_t stride)
{
    pcs_buf b{};
    b.ptr = ptr;
    b.kind = PCS_RING;
    b.row_bytes = row;
    b.capacity = cap;
    b.head = head;
    b.window = window;
    b.outer = outer;
    b.outer_stride = stride;
    return b;
}

// Physical address of logical byte L of a run list (the run with the largest
// lstart <= L).
static uint64_t address_of(const std::vector<Run> &rs, uint64_t L)
{
    size_t k = 0;
    while (k + 1 < rs.size() && rs[k + 1].lstart <= L) ++k;
    return rs[k].addr + (L - rs[k].lstart);
}

static void test_ring_runs(uint64_t seed)
{
    std::mt19937_64 rng(seed);
    for (int it = 0; it < 4000; ++it) {
        const uint64_t row = 16 * (1 + rng() % 300);
        const uint64_t cap = 1 + rng() % 40;
        const uint64_t head = rng() % cap;
        const uint64_t window = rng() % (cap + 1);
        const uint64_t outer = rng() % 6;
        // Strides: packed rings (adjacent, so runs can merge across rings) or gaps.
        const uint64_t stride = cap * row + 16 * (rng() % 3 == 0 ? 0 : rng() % 5);
        const uint64_t ptr = 16 * (1 + rng() % (1u << 20));
        const pcs_buf b = ring_buf(ptr, outer, cap, row, head, window, stride);
        Layout lay;
        std::vector<Run> rs;
        std::string why;
        CHECK(describe(b, 0, &lay, &rs, &why) == PCS_OK);
        const uint64_t total = outer * window * row;
        CHECK(lay.kind == PCS_RING && lay.nbytes == total);
        CHECK(lay.nchunks == (total + kChunk - 1) / kChunk);
        CHECK(lay.ngroups == (lay.nchunks + kGroupChunks - 1) / kGroupChunks);
        CHECK(lay.row_bytes == row && lay.window == window && lay.outer == outer);
        CHECK(!rs.empty() && rs[0].lstart == 0);
        CHECK(rs.size() <= std::max<uint64_t>(1, 2 * outer));
        for (size_t k = 1; k < rs.size(); ++k) {
            CHECK(rs[k].lstart > rs[k - 1].lstart);
            CHECK(rs[k].lstart < total);
            // Maximal: no run physically continues the previous one.
            CHECK(rs[k - 1].addr + (rs[k].lstart - rs[k - 1].lstart) != rs[k].addr);
            CHECK(rs[k].lstart % row == 0);  // runs break only at row boundaries
        }
        for (uint64_t o = 0; o < outer; ++o)
            for (uint64_t t = 0; t < window; ++t) {
                const uint64_t L = (o * window + t) * row;
                const uint64_t want = ptr + o * stride + ((head + t) % cap) * row;
                CHECK(address_of(rs, L) == want);
                CHECK(address_of(rs, L + row - 1) == want + row - 1);
            }
        // nbytes may be passed explicitly.
        pcs_buf b2 = b;
        b2.nbytes = total;
        std::vector<Run> rs2;
        CHECK(describe(b2, 0, &lay, &rs2, &why) == PCS_OK && rs2.size() == rs.size());
    }
}

static void test_flat_and_validation()
{
    Layout lay;
    std::vector<Run> rs;
    std::string why;
    // Valid flat buffers, including the empty one and a ragged size.
    CHECK(describe(flat_buf(0, 0), 0, &lay, &rs, &why) == PCS_OK && lay.nchunks == 0 && lay.ngroups == 0);
    rs.clear();
    CHECK(describe(flat_buf(4096, 1), 0, &lay, &rs, &why) == PCS_OK && lay.nchunks == 1 && rs.size() == 1);
    CHECK(rs[0].lstart == 0 && rs[0].addr == 4096);
    rs.clear();
    CHECK(describe(flat_buf(16, 64 * kChunk + 1), 0, &lay, &rs, &why) == PCS_OK);
    CHECK(lay.nchunks == 65 && lay.ngroups == 2);
    // A flat buffer reaching the top of the address space: its chunk count
    // does not wrap either.
    rs.clear();
    CHECK(describe(flat_buf(16, UINT64_MAX - 31), 0, &lay, &rs, &why) == PCS_OK);
    CHECK(lay.nchunks == (UINT64_MAX - 31) / kChunk + 1);
    // Valid degenerate rings: an empty window and no rings at all.
    rs.clear();
    CHECK(describe(ring_buf(256, 4, 8, 32, 3, 0, 256), 0, &lay, &rs, &why) == PCS_OK && lay.nbytes == 0);
    rs.clear();
    CHECK(describe(ring_buf(256, 0, 8, 32, 3, 5, 256), 0, &lay, &rs, &why) == PCS_OK && lay.nbytes == 0);
    // A full window (window == capacity) at a nonzero head wraps in every ring.
    rs.clear();
    CHECK(describe(ring_buf(1 << 20, 2, 8, 32, 5, 8, 1024), 0, &lay, &rs, &why) == PCS_OK && rs.size() == 4);

    struct Bad {
        pcs_buf b;
        const char *what;
    };
    pcs_buf flags = flat_buf(16, 16);
    flags.flags = 1;
    pcs_buf kind = flat_buf(16, 16);
    kind.kind = 7;
    pcs_buf wrong_n = ring_buf(256, 2, 8, 32, 0, 4, 256);
    wrong_n.nbytes = 2 * 4 * 32 + 16;
    const Bad bad[] = {
        {flags, "reserved flags"},
        {kind, "unknown kind"},
        {flat_buf(8, 16), "misaligned flat pointer"},
        {flat_buf(0, 16), "null flat pointer"},
        {flat_buf(UINT64_MAX - 15, 32), "flat range wraps"},
        {ring_buf(256, 1, 8, 0, 0, 4, 0), "zero row"},
        {ring_buf(256, 1, 8, 24, 0, 4, 0), "row not a multiple of 16"},
        {ring_buf(264, 1, 8, 32, 0, 4, 0), "misaligned ring pointer"},
        {ring_buf(256, 2, 8, 32, 0, 4, 264), "stride not a multiple of 16"},
        {ring_buf(256, 1, 0, 32, 0, 0, 0), "zero capacity"},
        {ring_buf(256, 1, 8, 32, 0, 9, 0), "window above capacity"},
        {ring_buf(256, 1, 8, 32, 8, 4, 0), "head at capacity"},
        {ring_buf(256, (1ULL << 30) + 1, 8, 32, 0, 4, 256), "too many rings"},
        {ring_buf(256, 2, 8, 32, 0, 4, 128), "rings overlap"},
        {wrong_n, "nbytes not outer*window*row"},
        {ring_buf(256, 1024, 1ULL << 30, 1ULL << 40, 0, 1ULL << 30, 0), "ring size overflows"},
        {ring_buf(0, 1, 8, 32, 0, 4, 0), "null ring pointer"},
        {ring_buf(UINT64_MAX - 255, 1, 8, 32, 0, 4, 0), "ring range wraps"},
        {ring_buf(1ULL << 63, 4, 8, 32, 0, 4, 1ULL << 62), "outer stride range wraps"},
    };
    for (const Bad &x : bad) {
        rs.clear();
        why.clear();
        const int st = describe(x.b, 3, &lay, &rs, &why);
        if (st != PCS_E_INVAL) fprintf(stderr, "accepted: %s\n", x.what);
        CHECK(st == PCS_E_INVAL);
        CHECK(rs.empty());                       // nothing appended on a rejection
        CHECK(why.find("buffer 3") == 0);        // the message names the buffer
    }
}

// ------------------------------------------------------------------ image header

struct Image {
    std::vector<Layout> lays;
    ImageLayout L;
    std::vector<uint8_t> bytes;
};

// Roots and fingerprints as an export writes them (nonzero words).
static void fill_hashes(std::vector<uint8_t> &img, const ImageLayout &L, uint64_t T)
{
    for (uint64_t i = L.roots_off; i < L.hashes_off + 8 * T; ++i) img[i] = (uint8_t)(0xA5 ^ (i * 29));
}

static Layout make_layout(std::mt19937_64 &rng)
{
    Layout y{};
    if (rng() % 2) {
        y.kind = PCS_FLAT;
        const uint64_t pick = rng() % 4;
        y.nbytes = pick == 0 ? 0 : pick == 1 ? 16 : rng() % 20000;
    } else {
        y.kind = PCS_RING;
        y.row_bytes = 16 * (1 + rng() % 40);
        y.window = rng() % 20;
        y.outer = rng() % 4;
        y.nbytes = y.row_bytes * y.window * y.outer;
    }
    y.nchunks = (y.nbytes + kChunk - 1) / kChunk;
    y.ngroups = (y.nchunks + kGroupChunks - 1) / kGroupChunks;
    return y;
}

static Image make_image(std::mt19937_64 &rng, uint32_t n)
{
    Image im;
    uint64_t T = 0, state = 0;
    for (uint32_t b = 0; b < n; ++b) {
        im.lays.push_back(make_layout(rng));
        T += im.lays.back().nchunks;
        state += im.lays.back().nbytes;
    }
    CHECK(image_layout(im.lays, T, &im.L));
    im.bytes.assign(im.L.size, 0xA5);
    write_image_header(im.bytes.data(), im.lays, T, state, im.L);
    fill_hashes(im.bytes, im.L, T);
    return im;
}

// Parses `n` bytes from a heap block of exactly that size, so a read past
// the end is caught by AddressSanitizer.
static int parse_exact(const uint8_t *src, uint64_t n, std::vector<Layout> *lays, ImageLayout *L)
{
    std::vector<uint8_t> copy(src, src + n);
    std::string why;
    const int st = parse_image_header(copy.data(), n, lays, L, &why);
    if (st) CHECK(!why.empty());
    return st;
}

// What an accepted header promises: every region it names lies in the image.
static void check_accepted(const std::vector<Layout> &lays, const ImageLayout &L, uint64_t size)
{
    const uint64_t n = lays.size();
    CHECK(L.roots_off == kImageHead + kImageDesc * n);
    CHECK(L.hashes_off == L.roots_off + 8 * (n + 1));
    CHECK(L.data_off % kAlign == 0 && L.data_off >= L.hashes_off);
    CHECK(L.data_off <= size && L.size == size && L.payload == size - L.data_off);
    uint64_t T = 0;
    for (size_t b = 0; b < n; ++b) {
        const Layout &y = lays[b];
        CHECK(y.kind == PCS_FLAT || y.kind == PCS_RING);
        CHECK(y.nchunks == (y.nbytes + kChunk - 1) / kChunk);
        CHECK(y.nbytes <= y.nchunks * kChunk);
        CHECK(L.comp_off[b] + y.nchunks * kChunk <= L.payload);
        T += y.nchunks;
    }
    CHECK(L.hashes_off + 8 * T <= L.data_off);
}

static void test_image_round_trip(uint64_t seed)
{
    std::mt19937_64 rng(seed);
    for (int it = 0; it < 300; ++it) {
        const Image im = make_image(rng, (uint32_t)(rng() % 7));
        std::vector<Layout> got;
        ImageLayout L;
        CHECK(parse_exact(im.bytes.data(), im.bytes.size(), &got, &L) == PCS_OK);
        CHECK(got.size() == im.lays.size());
        for (size_t b = 0; b < got.size(); ++b) {
            CHECK(got[b].kind == im.lays[b].kind && got[b].nbytes == im.lays[b].nbytes);
            CHECK(got[b].nchunks == im.lays[b].nchunks && got[b].ngroups == im.lays[b].ngroups);
            if (got[b].kind == PCS_RING)
                CHECK(got[b].row_bytes == im.lays[b].row_bytes && got[b].window == im.lays[b].window &&
                      got[b].outer == im.lays[b].outer);
            CHECK(L.comp_off[b] == im.L.comp_off[b]);
        }
        CHECK(L.roots_off == im.L.roots_off && L.hashes_off == im.L.hashes_off && L.data_off == im.L.data_off);
        CHECK(L.payload == im.L.payload && L.size == im.L.size);
        check_accepted(got, L, im.bytes.size());
    }
}

static void test_image_corruptions()
{
    std::mt19937_64 rng(7);
    // A fixed image with one flat buffer and one ring.
    Image im;
    Layout f{};
    f.kind = PCS_FLAT;
    f.nbytes = 5000;
    Layout r{};
    r.kind = PCS_RING;
    r.row_bytes = 64;
    r.window = 10;
    r.outer = 3;
    r.nbytes = 64 * 10 * 3;
    for (Layout *y : {&f, &r}) {
        y->nchunks = (y->nbytes + kChunk - 1) / kChunk;
        y->ngroups = 1;
        im.lays.push_back(*y);
    }
    const uint64_t T = f.nchunks + r.nchunks, state = f.nbytes + r.nbytes;
    CHECK(image_layout(im.lays, T, &im.L));
    im.bytes.assign(im.L.size, 0);
    write_image_header(im.bytes.data(), im.lays, T, state, im.L);
    fill_hashes(im.bytes, im.L, T);
    std::vector<Layout> got;
    ImageLayout L;
    CHECK(parse_exact(im.bytes.data(), im.bytes.size(), &got, &L) == PCS_OK);

    const uint64_t d0 = kImageHead, d1 = kImageHead + kImageDesc;
    struct Edit {
        uint64_t at;
        int width;  // 4 or 8
        uint64_t value;
        const char *what;
    };
    const Edit edits[] = {
        {0, 4, 0x534350ull, "magic"},
        {8, 4, 2, "version"},
        {12, 4, 3, "buffer count"},
        {12, 4, kImageMaxBufs + 1, "buffer count above the limit"},
        {16, 8, T + 1, "chunk total"},
        {24, 8, state + 1, "state bytes"},
        {32, 8, im.L.payload + kChunk, "payload bytes"},
        {40, 8, 1, "flags"},
        {d0, 4, 2, "kind"},
        {d0 + 4, 4, 1, "reserved word"},
        {d0 + 40, 8, 1, "reserved quad"},
        {d0 + 8, 8, 8000, "flat size (chunk count unchanged)"},
        {d0 + 16, 8, 16, "flat buffer with a row size"},
        {d1 + 16, 8, 0, "ring with a zero row"},
        {d1 + 16, 8, 72, "ring row not a multiple of 16"},
        {d1 + 24, 8, 11, "ring window inconsistent with its size"},
        {d1 + 32, 8, 1ULL << 62, "ring count overflowing its size"},
    };
    for (const Edit &e : edits) {
        std::vector<uint8_t> b = im.bytes;
        if (e.width == 4) put32(b.data() + e.at, (uint32_t)e.value);
        else put64(b.data() + e.at, e.value);
        const int st = parse_exact(b.data(), b.size(), &got, &L);
        if (st != PCS_E_CORRUPT) fprintf(stderr, "accepted: %s\n", e.what);
        CHECK(st == PCS_E_CORRUPT);
    }
    // Truncated and extended images, and sizes below the fixed header.
    for (uint64_t cut : {(uint64_t)1, (uint64_t)kChunk, (uint64_t)im.bytes.size() - kImageHead})
        CHECK(parse_exact(im.bytes.data(), im.bytes.size() - cut, &got, &L) == PCS_E_CORRUPT);
    for (uint64_t n : {(uint64_t)0, (uint64_t)8, kImageHead - 1})
        CHECK(parse_exact(im.bytes.data(), n, &got, &L) == PCS_E_CORRUPT);
    std::vector<uint8_t> longer = im.bytes;
    longer.resize(longer.size() + kChunk, 0);
    CHECK(parse_exact(longer.data(), longer.size(), &got, &L) == PCS_E_CORRUPT);

    // A size near 2^64 whose chunk count would wrap to 0 under (n + 4095) / 4096,
    // with totals set to match that wrapped reading: must be refused, not
    // accepted as an empty payload of an enormous buffer.
    {
        std::vector<Layout> one(1);
        one[0].kind = PCS_FLAT;
        ImageLayout L1;
        CHECK(image_layout(one, 0, &L1));
        std::vector<uint8_t> b(L1.size, 0);
        write_image_header(b.data(), one, 0, 0, L1);
        put64(b.data() + kImageHead + 8, UINT64_MAX);  // nbytes
        put64(b.data() + 24, UINT64_MAX);              // state bytes
        CHECK(parse_exact(b.data(), b.size(), &got, &L) == PCS_E_CORRUPT);
        put64(b.data() + kImageHead + 8, UINT64_MAX - 4094);
        put64(b.data() + 24, UINT64_MAX - 4094);
        CHECK(parse_exact(b.data(), b.size(), &got, &L) == PCS_E_CORRUPT);
    }

    // Random mutations of the header and descriptors, and random truncations:
    // never a read outside the image; anything accepted is self-consistent.
    int accepted = 0;
    for (int it = 0; it < 20000; ++it) {
        std::vector<uint8_t> b = im.bytes;
        const int flips = 1 + (int)(rng() % 4);
        for (int k = 0; k < flips; ++k) {
            const uint64_t at = rng() % (im.L.hashes_off + 16);
            b[at] = (uint8_t)rng();
        }
        uint64_t size = b.size();
        if (rng() % 4 == 0) size = rng() % (b.size() + 1);
        if (parse_exact(b.data(), size, &got, &L) == PCS_OK) {
            ++accepted;
            check_accepted(got, L, size);
        }
    }
    CHECK(accepted < 20000);
}

// ------------------------------------------------------------- tile order

// xcd_tile_of (pcs_layout.h) is a bijection of [0, nb), and workgroup b
// (XCD b mod 8, position b / 8 there) gets a tile of its XCD's share: below
// 16384 tiles the XCD's contiguous eighth, walked in order from a start
// staggered by x/8 of its length; from 16384 tiles the 512-tile blocks dealt
// to that XCD, walked in order, with the tail of fewer than eight blocks in
// launch order.
static void test_tile_order()
{
    std::vector<uint32_t> sizes;
    for (uint32_t nb = 1; nb <= 300; ++nb) sizes.push_back(nb);
    for (uint32_t nb : {1023u, 1024u, 1025u, 2047u, 2048u, 2049u, 4096u, 8191u, 16383u, 16384u, 16385u, 16391u,
                        16392u, 20000u, 20480u, 24575u, 36864u, 65535u, 65536u, 137216u, 271536u})
        sizes.push_back(nb);
    for (uint32_t nb : sizes) {
        std::vector<uint8_t> seen(nb, 0);
        for (uint32_t b = 0; b < nb; ++b) {
            const uint32_t t = xcd_tile_of(b, nb);
            CHECK(t < nb);
            if (t >= nb) continue;
            CHECK(!seen[t]);
            seen[t] = 1;
            const uint32_t x = b % kXcds, i = b / kXcds;
            if (nb < kXcdBlockJobs) {
                const uint32_t per = nb / kXcds, rem = nb % kXcds, n = per + (x < rem ? 1 : 0);
                const uint32_t lo = x * per + (x < rem ? x : rem);
                CHECK(t >= lo && t < lo + n);                               // in the XCD's eighth
                CHECK(t - lo == (i + x * (n / kXcds)) % n);                 // walked from the staggered start
            } else {
                const uint32_t full = nb / (kXcds * kXcdBlock);
                if (b >= full * kXcds * kXcdBlock) {
                    CHECK(t == b);                                          // the tail keeps the launch order
                } else {
                    CHECK((t / kXcdBlock) % kXcds == x);                    // a block dealt to this XCD
                    CHECK(t / kXcdBlock / kXcds == i / kXcdBlock && t % kXcdBlock == i % kXcdBlock);
                }
            }
        }
    }
}

int main()
{
    test_tile_order();
    for (uint64_t s = 1; s <= 12; ++s) test_arena(s);
    test_ring_runs(3);
    test_flat_and_validation();
    test_image_round_trip(5);
    test_image_corruptions();
    printf("ok %d checks\n", g_checks);
    return 0;
}

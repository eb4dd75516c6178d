// pcs_host.h -- host-side logic of libpcs that needs no GPU: the arena
// sub-allocator, plan descriptors resolved into physical runs, and the
// snapshot image header.  Header-only so that the runtime and a host-only
// test program build it the same way.  Internal to the library (not part of
// the C ABI).
#pragma once

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "../../include/pcs.h"
#include "pcs_layout.h"

namespace pcs {

constexpr uint64_t kAlign = 4096;

inline uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }
// ceil(x / a) without the wrap of (x + a - 1) / a near 2^64.
inline uint64_t div_up(uint64_t x, uint64_t a) { return x / a + (x % a != 0); }
inline bool mul_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_mul_overflow(a, b, out); }
inline bool add_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_add_overflow(a, b, out); }

inline void set_err(std::string *err, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
inline void set_err(std::string *err, const char *fmt, ...)
{
    if (!err) return;
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    *err = buf;
}

// First-fit allocator over [0, size) in 4096-byte units.
class Arena {
  public:
    void init(uint64_t size)
    {
        size_ = size;
        used_ = 0;
        free_.clear();
        if (size) free_[0] = size;
    }
    bool alloc(uint64_t bytes, uint64_t *off)
    {
        if (!units(bytes, &bytes)) return false;
        for (auto it = free_.begin(); it != free_.end(); ++it) {
            if (it->second < bytes) continue;
            *off = it->first;
            const uint64_t rest = it->second - bytes, noff = it->first + bytes;
            free_.erase(it);
            if (rest) free_[noff] = rest;
            used_ += bytes;
            return true;
        }
        return false;
    }
    // Highest-address fit: [end - bytes, end) of the highest free range that
    // holds it.  Incremental payload reservations come from the top, so the
    // part a reservation gives back (its low end) merges with free space.
    bool alloc_top(uint64_t bytes, uint64_t *off)
    {
        if (!units(bytes, &bytes)) return false;
        for (auto it = free_.rbegin(); it != free_.rend(); ++it) {
            if (it->second < bytes) continue;
            const uint64_t start = it->first, size = it->second;
            *off = start + size - bytes;
            if (size == bytes) free_.erase(start);
            else free_[start] = size - bytes;
            used_ += bytes;
            return true;
        }
        return false;
    }
    // Returns [off, off + bytes) (rounded as at allocation) to the free map.
    void release(uint64_t off, uint64_t bytes)
    {
        units(bytes, &bytes);
        used_ -= bytes;
        auto it = free_.emplace(off, bytes).first;
        auto nx = std::next(it);
        if (nx != free_.end() && it->first + it->second == nx->first) {
            it->second += nx->second;
            free_.erase(nx);
        }
        if (it != free_.begin()) {
            auto pv = std::prev(it);
            if (pv->first + pv->second == it->first) {
                pv->second += it->second;
                free_.erase(it);
            }
        }
    }
    uint64_t used() const { return used_; }
    uint64_t size() const { return size_; }
    uint64_t largest() const
    {
        uint64_t m = 0;
        for (auto &kv : free_) m = std::max(m, kv.second);
        return m;
    }
    const std::map<uint64_t, uint64_t> &free_ranges() const { return free_; }

  private:
    // Rounds a request up to whole 4096-byte units (at least one); false if
    // that does not fit in 64 bits (no arena can hold it).
    static bool units(uint64_t bytes, uint64_t *out)
    {
        if (bytes > UINT64_MAX - (kAlign - 1)) return false;
        *out = std::max<uint64_t>(kAlign, round_up(bytes, kAlign));
        return true;
    }
    uint64_t size_ = 0, used_ = 0;
    std::map<uint64_t, uint64_t> free_;
};

// A plan buffer resolved into its logical byte stream.
struct Layout {
    uint32_t kind;
    uint64_t nbytes, nchunks, ngroups;
    uint64_t row_bytes, window, outer;  // RING shape (restore compatibility)
};

// Validates one descriptor and appends its runs (logical start, physical
// address), merging physically adjacent pieces.  PCS_OK, or PCS_E_INVAL with
// the reason in *err.  Every address a run covers lies in
// [ptr, ptr + extent) without wrapping 64 bits.
inline int describe(const pcs_buf &b, uint32_t idx, Layout *lay, std::vector<Run> *runs, std::string *err)
{
    if (b.flags != 0) return set_err(err, "buffer %u: flags must be 0", idx), PCS_E_INVAL;
    Layout L{};
    L.kind = b.kind;
    std::vector<Run> rs;
    if (b.kind == PCS_FLAT) {
        if (b.nbytes && (b.ptr == 0 || b.ptr % 16))
            return set_err(err, "buffer %u: flat ptr must be non-null and 16-byte aligned", idx), PCS_E_INVAL;
        if (b.ptr > UINT64_MAX - b.nbytes)
            return set_err(err, "buffer %u: address range wraps", idx), PCS_E_INVAL;
        L.nbytes = b.nbytes;
        rs.push_back({0, b.ptr});
    } else if (b.kind == PCS_RING) {
        if (b.row_bytes == 0 || b.row_bytes % 16 || b.ptr % 16 || b.outer_stride % 16)
            return set_err(err, "buffer %u: ring ptr, row_bytes and outer_stride must be multiples of 16", idx),
                   PCS_E_INVAL;
        if (b.capacity == 0 || b.window > b.capacity || b.head >= b.capacity)
            return set_err(err, "buffer %u: ring needs 0 <= window <= capacity and head < capacity", idx),
                   PCS_E_INVAL;
        if (b.outer > (1ULL << 30)) return set_err(err, "buffer %u: too many rings", idx), PCS_E_INVAL;
        uint64_t ring_span, win_bytes, total, extent = 0;
        if (!mul_ok(b.capacity, b.row_bytes, &ring_span) || !mul_ok(b.window, b.row_bytes, &win_bytes) ||
            !mul_ok(win_bytes, b.outer, &total))
            return set_err(err, "buffer %u: ring size overflows", idx), PCS_E_INVAL;
        if (b.outer > 1 && b.outer_stride < ring_span)
            return set_err(err, "buffer %u: outer_stride < capacity*row_bytes (rings overlap)", idx), PCS_E_INVAL;
        if (b.nbytes != 0 && b.nbytes != total)
            return set_err(err, "buffer %u: ring nbytes must be 0 or outer*window*row_bytes", idx), PCS_E_INVAL;
        if (total && b.ptr == 0) return set_err(err, "buffer %u: null ring pointer", idx), PCS_E_INVAL;
        if (total && (!mul_ok(b.outer - 1, b.outer_stride, &extent) || !add_ok(extent, ring_span, &extent) ||
                      b.ptr > UINT64_MAX - extent))
            return set_err(err, "buffer %u: address range wraps", idx), PCS_E_INVAL;
        L.nbytes = total;
        L.row_bytes = b.row_bytes;
        L.window = b.window;
        L.outer = b.outer;
        uint64_t lpos = 0;
        auto add = [&](uint64_t addr, uint64_t len) {
            if (len == 0) return;
            if (!rs.empty()) {
                const Run &p = rs.back();
                if (p.addr + (lpos - p.lstart) == addr) {  // physically continues the previous run
                    lpos += len;
                    return;
                }
            }
            rs.push_back({lpos, addr});
            lpos += len;
        };
        for (uint64_t o = 0; o < b.outer && total; ++o) {
            const uint64_t base = b.ptr + o * b.outer_stride;
            const uint64_t first = std::min(b.window, b.capacity - b.head);
            add(base + b.head * b.row_bytes, first * b.row_bytes);
            add(base, (b.window - first) * b.row_bytes);
        }
        if (rs.empty()) rs.push_back({0, b.ptr});
    } else {
        return set_err(err, "buffer %u: unknown kind %u", idx, b.kind), PCS_E_INVAL;
    }
    L.nchunks = div_up(L.nbytes, kChunk);
    L.ngroups = div_up(L.nchunks, kGroupChunks);
    *lay = L;
    runs->insert(runs->end(), rs.begin(), rs.end());
    return PCS_OK;
}

// ---------------------------------------------------------------- snapshot images
//
// A self-contained host image of a snapshot (little-endian):
//   [0, 8)    magic "PCSIMG01"
//   [8, 12)   u32 version (1)         [12, 16)  u32 nbufs n
//   [16, 24)  u64 total chunks T      [24, 32)  u64 state bytes
//   [32, 40)  u64 payload bytes       [40, 48)  u64 flags (0)
//   n x 48 B  per buffer: u32 kind, u32 0, u64 nbytes, u64 row_bytes,
//             u64 window, u64 outer, u64 0   (ring fields 0 for flat buffers)
//   (n+1) x 8 buffer roots, then the session root
//   T x 8     chunk fingerprints, buffer-major
//   zero padding to a 4096-byte boundary, then the payload in the canonical
//   full-snapshot layout (components 4096-aligned, zero padded).
constexpr char kImageMagic[8] = {'P', 'C', 'S', 'I', 'M', 'G', '0', '1'};
constexpr uint64_t kImageHead = 48, kImageDesc = 48;
constexpr uint32_t kImageMaxBufs = 1u << 24;

struct ImageLayout {
    uint64_t roots_off, hashes_off, data_off, size, payload;
    std::vector<uint64_t> comp_off;
};

inline void put32(uint8_t *p, uint32_t v) { memcpy(p, &v, 4); }
inline void put64(uint8_t *p, uint64_t v) { memcpy(p, &v, 8); }
inline uint32_t get32(const uint8_t *p)
{
    uint32_t v;
    memcpy(&v, p, 4);
    return v;
}
inline uint64_t get64(const uint8_t *p)
{
    uint64_t v;
    memcpy(&v, p, 8);
    return v;
}

// Offsets of an image over buffers `bufs` holding T chunks in total; false
// if any offset does not fit in 64 bits.
inline bool image_layout(const std::vector<Layout> &bufs, uint64_t T, ImageLayout *L)
{
    const uint64_t n = bufs.size();
    uint64_t t;
    L->comp_off.clear();
    L->roots_off = kImageHead + kImageDesc * n;  // n <= kImageMaxBufs: no overflow
    L->hashes_off = L->roots_off + 8 * (n + 1);
    if (!mul_ok(T, 8, &t) || !add_ok(L->hashes_off, t, &t) || t > UINT64_MAX - kAlign) return false;
    L->data_off = round_up(t, kAlign);
    L->payload = 0;
    for (auto &b : bufs) {
        L->comp_off.push_back(L->payload);
        if (!mul_ok(b.nchunks, kChunk, &t) || !add_ok(L->payload, t, &L->payload)) return false;
    }
    return add_ok(L->data_off, L->payload, &L->size);
}

// Writes the header, descriptors and zero padding of an image (everything
// before the roots is written; roots, fingerprints and payload are the
// caller's).  img holds at least L.data_off bytes.
inline void write_image_header(uint8_t *img, const std::vector<Layout> &bufs, uint64_t T, uint64_t state_bytes,
                               const ImageLayout &L)
{
    memset(img, 0, L.data_off);
    memcpy(img, kImageMagic, 8);
    put32(img + 8, 1);
    put32(img + 12, (uint32_t)bufs.size());
    put64(img + 16, T);
    put64(img + 24, state_bytes);
    put64(img + 32, L.payload);
    for (size_t b = 0; b < bufs.size(); ++b) {
        uint8_t *d = img + kImageHead + kImageDesc * b;
        const Layout &y = bufs[b];
        put32(d, y.kind);
        put64(d + 8, y.nbytes);
        put64(d + 16, y.kind == PCS_RING ? y.row_bytes : 0);
        put64(d + 24, y.kind == PCS_RING ? y.window : 0);
        put64(d + 32, y.kind == PCS_RING ? y.outer : 0);
    }
}

// Parses and checks the header of an image of `size` bytes.  On PCS_OK,
// *lays and *L describe it and every region they name (roots, fingerprints,
// each buffer's payload component) lies inside [0, size).  Anything
// inconsistent is PCS_E_CORRUPT with the reason in *err.
inline int parse_image_header(const uint8_t *img, uint64_t size, std::vector<Layout> *lays, ImageLayout *L,
                              std::string *err)
{
    if (size < kImageHead || memcmp(img, kImageMagic, 8) != 0)
        return set_err(err, "not a snapshot image"), PCS_E_CORRUPT;
    if (get32(img + 8) != 1) return set_err(err, "unknown image version %u", get32(img + 8)), PCS_E_CORRUPT;
    const uint32_t n = get32(img + 12);
    const uint64_t T = get64(img + 16), state = get64(img + 24), payload = get64(img + 32);
    if (get64(img + 40) != 0) return set_err(err, "unknown image flags"), PCS_E_CORRUPT;
    if (n > kImageMaxBufs || size - kImageHead < kImageDesc * (uint64_t)n)
        return set_err(err, "truncated image header"), PCS_E_CORRUPT;
    lays->assign(n, Layout{});
    uint64_t sum_chunks = 0, sum_bytes = 0;
    for (uint32_t b = 0; b < n; ++b) {
        const uint8_t *d = img + kImageHead + kImageDesc * b;
        Layout y{};
        y.kind = get32(d);
        y.nbytes = get64(d + 8);
        y.row_bytes = get64(d + 16);
        y.window = get64(d + 24);
        y.outer = get64(d + 32);
        if (get32(d + 4) != 0 || get64(d + 40) != 0)
            return set_err(err, "buffer %u: reserved fields are not 0", b), PCS_E_CORRUPT;
        if (y.kind == PCS_FLAT) {
            if (y.row_bytes || y.window || y.outer)
                return set_err(err, "buffer %u: flat buffer with ring fields", b), PCS_E_CORRUPT;
        } else if (y.kind == PCS_RING) {
            uint64_t t;
            if (y.row_bytes == 0 || y.row_bytes % 16 || !mul_ok(y.window, y.row_bytes, &t) ||
                !mul_ok(t, y.outer, &t) || t != y.nbytes)
                return set_err(err, "buffer %u: ring shape does not match its size", b), PCS_E_CORRUPT;
        } else {
            return set_err(err, "buffer %u: bad kind %u", b, y.kind), PCS_E_CORRUPT;
        }
        // A payload component holds nbytes, so nbytes <= size in any real image
        // (the final size check implies it too; this bounds the sums early).
        if (y.nbytes > size) return set_err(err, "buffer %u: larger than the image", b), PCS_E_CORRUPT;
        y.nchunks = div_up(y.nbytes, kChunk);
        y.ngroups = div_up(y.nchunks, kGroupChunks);
        if (!add_ok(sum_chunks, y.nchunks, &sum_chunks) || !add_ok(sum_bytes, y.nbytes, &sum_bytes))
            return set_err(err, "image sizes overflow"), PCS_E_CORRUPT;
        (*lays)[b] = y;
    }
    if (!image_layout(*lays, sum_chunks, L)) return set_err(err, "image sizes overflow"), PCS_E_CORRUPT;
    if (sum_chunks != T || sum_bytes != state || L->payload != payload || L->size != size)
        return set_err(err, "image header is inconsistent with its size"), PCS_E_CORRUPT;
    return PCS_OK;
}

}  // namespace pcs

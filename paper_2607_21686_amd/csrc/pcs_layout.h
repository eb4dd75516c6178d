// pcs_layout.h -- descriptors and constants shared by the host runtime and
// the gfx950 kernels of libpcs: plain structs with fixed layouts, no HIP.
// Internal to the library (not part of the C ABI).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace pcs {

constexpr uint64_t kChunk = 4096;       // fingerprint and snapshot granule (bytes)
constexpr uint32_t kGroupChunks = 64;   // chunks per work group and per bitmap word

// A maximal physically contiguous piece of a buffer's logical byte stream:
// logical bytes [lstart, next run's lstart) live at addr onwards.  A flat
// buffer is one run; a ring window is at most two runs per ring (before and
// after the wrap), merged where physically adjacent.
struct Run {
    uint64_t lstart;
    uint64_t addr;
};

// One buffer of a job.  Every kernel grids over 64-chunk groups of one
// buffer; group_begin is this buffer's first group in the job.
struct JobBuf {
    uint64_t nbytes;          // logical bytes
    uint64_t nchunks;         // ceil(nbytes / 4096)
    uint64_t chunk_begin;     // first chunk of this buffer in job-wide chunk order
    uint64_t group_begin;     // first 64-chunk group of this buffer in the job
    uint64_t payload;         // device address of chunk 0's 4096-byte slot (pack dst, restore src)
    uint64_t manifest;        // restore: device address of uint64 arena offsets, one per chunk
                              // incremental pack: where this buffer's new manifest entries go
    uint64_t hash_dst[2];     // device addresses of chunk 0's fingerprint outputs (0 = none)
    uint64_t root_dst[2];     // device addresses of the root outputs (0 = none)
    uint64_t parent_hash;     // incremental: device address of the parent's chunk-0 fingerprint;
                              // verified restore: of the snapshot's stored chunk-0 fingerprint
    uint64_t parent_chunks;   // incremental: chunks the parent held for this buffer
    uint64_t parent_manifest; // incremental: parent's manifest entries (0 if the parent is full)
    uint64_t parent_slot0;    // incremental, full parent: arena offset of the parent's chunk-0 slot
    uint32_t run_begin;       // this buffer's runs in the job's run table
    uint32_t run_count;
    uint32_t pad[2];
};
static_assert(sizeof(JobBuf) == 128, "JobBuf layout");

// A list reduced by the Merkle kernel: values [begin, begin + count) of the
// input array; the root goes to dst[0] / dst[1] (0 = none) and scratch[idx].
struct MerkleList {
    uint64_t begin;
    uint64_t count;
    uint64_t dst[2];
};

// Where a launch finds its buffer and run tables.
//   DevTables: in device memory (uploaded per call), with a group map
//              written by k_group_map that gives each group its buffer and
//              the run holding its first byte; any job size.
//   ArgTables: carried in the kernel arguments themselves (no upload, no map
//              kernel: a workgroup finds its buffer and first run with short
//              searches); jobs of at most kArgBufs buffers and kArgRuns runs.
constexpr uint32_t kArgBufs = 16, kArgRuns = 64;
// Small jobs (at most kSmallJobGroups groups) are cut into kSmallTiles
// sub-tiles per group, so that a few groups still spread over many CUs.
// Fingerprint and pack tiles then write one Merkle node per sub-tile (an
// aligned 8-chunk subtree, which the Merkle lists reduce like group nodes).
// Smaller tiles do not pay: a tile's fingerprint is bounded by one chunk's
// XXH64 chain (128 dependent rounds per accumulator), which 8-chunk tiles
// overlap with their loads.
constexpr uint64_t kSmallJobGroups = 128;
constexpr uint32_t kSmallTiles = 8;
inline uint32_t tile_split(uint64_t ngroups) { return ngroups <= kSmallJobGroups ? kSmallTiles : 1; }
struct GroupRef {
    uint32_t buf;
    uint32_t run;
};

// Tile order of the tile kernels: the tile workgroup b of a launch of nb
// workgroups takes.  The dispatcher deals a launch's workgroups to the eight
// XCDs in turn (workgroup b runs on XCD b mod 8), so the tiles are handed
// out XCD by XCD:
//   - below kXcdBlockJobs tiles: XCD x works through the x-th contiguous
//     eighth of the job in order, entered at a point staggered by x/8 of its
//     length (wrapping), so that the eight streams do not walk over the same
//     memory channels in step;
//   - from kXcdBlockJobs tiles: blocks of kXcdBlock consecutive tiles are
//     dealt to the XCDs in turn, so every XCD streams through every part of
//     the job and none is left with a stretch of memory that happens to be
//     slower; the tail of fewer than eight blocks keeps the launch order.
// A bijection of [0, nb).  (constexpr: callable from host and device code.)
constexpr uint32_t kXcds = 8, kXcdBlock = 512, kXcdBlockJobs = 16384;
constexpr uint32_t xcd_tile_of(uint32_t b, uint32_t nb)
{
    const uint32_t x = b % kXcds, i = b / kXcds;
    if (nb >= kXcdBlockJobs) {
        const uint32_t full = nb / (kXcds * kXcdBlock);  // whole rounds of blocks
        if (b >= full * kXcds * kXcdBlock) return b;
        return ((i / kXcdBlock) * kXcds + x) * kXcdBlock + i % kXcdBlock;
    }
    const uint32_t per = nb / kXcds, rem = nb % kXcds;
    const uint32_t n = per + (x < rem ? 1u : 0u);  // tiles of XCD x (>= 1 when workgroup b exists)
    return x * per + (x < rem ? x : rem) + (i + x * (n / kXcds)) % n;
}

struct DevTables {
    const JobBuf *bufs;
    const Run *runs;
    const GroupRef *map;
    uint32_t nbuf;
    uint32_t pad;
};
struct ArgTables {
    uint32_t nbuf;
    uint32_t pad;
    JobBuf bufs[kArgBufs];
    Run runs[kArgRuns];
};
// Kernel arguments are limited to 4 KiB; a launch passes one ArgTables and at
// most a few pointers and sizes besides.
static_assert(sizeof(ArgTables) + 256 <= 4096, "argument tables must fit in the kernel arguments");
// Merkle lists carried in the kernel arguments: the first nbuf_lists reduce
// group nodes to buffer roots, the rest reduce those roots to session roots
// (their begin/count index the buffer lists).
struct ArgLists {
    uint32_t nbuf_lists;
    uint32_t nlists;
    MerkleList lists[kArgBufs + 1];
};
static_assert(sizeof(ArgLists) + 256 <= 4096, "Merkle lists must fit in the kernel arguments");
// The small incremental launch passes both, with a few pointers and sizes.
static_assert(sizeof(ArgLists) + sizeof(ArgTables) + 128 <= 4096, "Merkle lists and tables must fit together");

// Buffer lists of a Merkle launch that hold more than kMerkleLdsValues
// values (a buffer of more than 1 GiB): when at most kLongLists of them, a
// grid-wide pass reduces their aligned 64-value blocks first,
// one wavefront each, into the list's first scratch level (at the list's own
// offset), and the per-list reduction starts from there.  Block b of the
// pass belongs to list j when block_begin[j] <= b < block_begin[j + 1].
constexpr uint64_t kMerkleLdsValues = 4096;
constexpr uint32_t kLongLists = 4;  // more long lists reduce in parallel, one workgroup each, anyway
struct LongLists {
    uint32_t n;
    uint32_t pad;
    uint64_t begin[kLongLists];
    uint64_t count[kLongLists];
    uint64_t block_begin[kLongLists + 1];
};

// The entry moves of a bank shrink, every part in one launch.  Part p moves
// the kept entries of entry_bytes eb from src to dst (stage: in place, the
// staging area for entries the compaction would overwrite before reading
// them; 0 out of place) in g-byte granules (16, 4 or 1, what the addresses
// and eb allow), spe slices of 256 granules per entry; its work items are
// [item_begin, item_begin + keep * spe).
struct ShrinkPart {
    uint64_t src, dst, stage;
    uint64_t eb;
    uint64_t item_begin;
    uint64_t g, spe;
};
constexpr uint32_t kShrinkParts = 64;
struct ShrinkParts {
    uint32_t n;
    uint32_t pad;
    uint64_t items;
    ShrinkPart p[kShrinkParts];
};
static_assert(sizeof(ShrinkParts) + 64 <= 4096, "shrink parts must fit in the kernel arguments");

}  // namespace pcs

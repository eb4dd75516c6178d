// pcs_device.h -- descriptors shared by the host runtime and the gfx950
// kernels of libpcs.  Internal to the library (not part of the C ABI).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

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
constexpr uint32_t kArgBufs = 8, kArgRuns = 64;
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
// Merkle lists carried in the kernel arguments: the first nbuf_lists reduce
// group nodes to buffer roots, the rest reduce those roots to session roots
// (their begin/count index the buffer lists).
struct ArgLists {
    uint32_t nbuf_lists;
    uint32_t nlists;
    MerkleList lists[kArgBufs + 1];
};

// Kernel launchers (pcs_kernels.hip).  All are asynchronous on `s`.
enum TileMode : int {
    kModeHash = 0,    // fingerprint the buffer's runs
    kModePack = 1,    // ... and store every chunk to its snapshot slot (checkpoint)
    kModeDiff = 2,    // ... and mark chunks new or changed against the parent (incremental)
    kModeVerify = 3,  // copy snapshot slots to the buffer's runs (restore), fingerprint
                      // the restored bytes and mark chunks whose fingerprint differs
                      // from the one stored at checkpoint time
};
hipError_t launch_group_map(const JobBuf *bufs, const Run *runs, uint32_t nbuf, uint64_t ngroups, GroupRef *map,
                            hipStream_t s);
template <class Tab>
hipError_t launch_tile(const Tab &tab, uint64_t ngroups, int mode, uint64_t *nodes, uint32_t *flag_count,
                       uint64_t *flag_mask, uint64_t arena_base, hipStream_t s, uint32_t tiles_per_group = 1);
template <class Tab>
hipError_t launch_copy(const Tab &tab, uint64_t ngroups, bool pack, uint64_t arena_base, hipStream_t s);
template <class Tab>
hipError_t launch_compact(const Tab &tab, uint64_t ngroups, const uint64_t *dirty_mask, const uint64_t *offsets,
                          uint64_t payload_arena_top, uint64_t *list, hipStream_t s);
template <class Tab>
hipError_t launch_pack_dirty(const Tab &tab, const uint64_t *list, const uint64_t *total, uint64_t max_slots,
                             uint64_t payload_top, hipStream_t s);
template <class Tab>
hipError_t launch_classify(const Tab &tab, uint64_t ngroups, const uint64_t *hashes, uint32_t K, uint64_t total,
                           uint64_t *bitmap, hipStream_t s);
template <class Tab>
hipError_t launch_labels(const Tab &tab, const uint64_t *bitmap, uint8_t *labels, hipStream_t s);
hipError_t launch_merkle(const MerkleList *lists, uint32_t nlists, const uint64_t *in,
                         uint64_t *scratch_a, uint64_t *scratch_b, uint64_t *roots_out,
                         hipStream_t s);
hipError_t launch_merkle_small(const ArgLists &lists, const uint64_t *in, uint64_t *scratch_a,
                               uint64_t *scratch_b, hipStream_t s);
hipError_t launch_scan(const uint32_t *counts, uint64_t n, uint64_t *offsets, uint64_t *total, hipStream_t s,
                       uint64_t *total_host = nullptr);
constexpr uint64_t kScanCompactMaxGroups = 4096;
// Small incremental jobs of at most this many groups scan and compact in one
// workgroup (one launch); larger ones scan in one workgroup and compact with
// one workgroup per group.
constexpr uint64_t kScanCompactFusedGroups = 16;
hipError_t launch_scan_compact_small(const ArgTables &tab, uint64_t ngroups, const uint32_t *counts,
                                     const uint64_t *dirty_mask, uint64_t payload_arena_top, uint64_t *list,
                                     uint64_t *total, uint64_t *total_host, hipStream_t s);
hipError_t launch_reverse_slots(uint64_t top, uint64_t dst, uint64_t n, hipStream_t s);
// Flips the lowest bit of the byte at device address addr.
hipError_t launch_flip_bit(uint64_t addr, hipStream_t s);
// Bank shrink: flags[i] = entry i is among the `keep` best-ranked (score
// order of pcs_bank_shrink), offsets = exclusive scan of flags, kept = the
// kept indices in increasing order.
hipError_t launch_shrink_select(const float *scores, uint32_t n, uint32_t keep, uint32_t *flags, uint64_t *offsets,
                                uint64_t *total, uint32_t *kept, hipStream_t s);
// dst entry j <- src entry kept[j] (entry j when kept is null), count entries
// of entry_bytes bytes.
hipError_t launch_gather_entries(uint64_t src, uint64_t dst, uint64_t entry_bytes, const uint32_t *kept,
                                 uint64_t count, hipStream_t s);

}  // namespace pcs

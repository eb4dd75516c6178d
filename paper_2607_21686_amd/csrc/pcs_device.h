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

// Kernel launchers (pcs_kernels.hip).  All are asynchronous on `s`.
hipError_t launch_group_map(const JobBuf *bufs, uint32_t nbuf, uint64_t ngroups, uint32_t *map,
                            hipStream_t s);
hipError_t launch_hash(const JobBuf *bufs, const Run *runs, const uint32_t *map, uint64_t ngroups,
                       bool copy, bool diff, uint64_t *nodes, uint32_t *dirty_count,
                       uint64_t *dirty_mask, hipStream_t s);
hipError_t launch_restore_verify(const JobBuf *bufs, const Run *runs, const uint32_t *map, uint64_t ngroups,
                                 uint64_t arena_base, uint64_t *bad_bitmap, hipStream_t s);
hipError_t launch_merkle(const MerkleList *lists, uint32_t nlists, const uint64_t *in,
                         uint64_t *scratch_a, uint64_t *scratch_b, uint64_t *roots_out,
                         hipStream_t s);
hipError_t launch_pack(const JobBuf *bufs, const Run *runs, const uint32_t *map, uint64_t ngroups,
                       hipStream_t s);
hipError_t launch_restore(const JobBuf *bufs, const Run *runs, const uint32_t *map,
                          uint64_t ngroups, uint64_t arena_base, hipStream_t s);
hipError_t launch_scan(const uint32_t *counts, uint64_t n, uint64_t *offsets, uint64_t *total,
                       hipStream_t s);
hipError_t launch_compact(const JobBuf *bufs, const uint32_t *map, uint64_t ngroups,
                          const uint64_t *dirty_mask, const uint64_t *offsets,
                          uint64_t payload_arena_top, uint64_t *list, hipStream_t s);
hipError_t launch_pack_dirty(const JobBuf *bufs, const Run *runs, const uint64_t *list,
                             const uint64_t *total, uint64_t max_slots, uint64_t payload_top,
                             hipStream_t s);
hipError_t launch_reverse_slots(uint64_t top, uint64_t dst, uint64_t n, hipStream_t s);
hipError_t launch_classify(const JobBuf *bufs, const uint32_t *map, uint64_t ngroups,
                           const uint64_t *hashes, uint32_t K, uint64_t total, uint64_t *bitmap,
                           hipStream_t s);
hipError_t launch_labels(const JobBuf *bufs, uint32_t nbuf, const uint64_t *bitmap,
                         uint8_t *labels, hipStream_t s);

}  // namespace pcs

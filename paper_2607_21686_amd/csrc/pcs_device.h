// pcs_device.h -- the gfx950 kernel launchers of libpcs (pcs_kernels.hip),
// over the descriptors of pcs_layout.h.  Internal to the library (not part
// of the C ABI).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "pcs_layout.h"

namespace pcs {

// Size of the per-device scratch array of the allocation-free fingerprint
// entry point, and its device address on the current device (valid for the
// life of the process; call once per device with that device current).
constexpr uint64_t kStaticScratchBytes = 16ULL << 20;
hipError_t static_scratch_address(uint64_t *addr);

// Dispatch timing: the next kernel launched by a launcher on this thread
// takes `start` and `stop` and stamps them with its own begin and end times.
// take_kernel_events_used() says whether a kernel took them (a launcher with
// no work launches none) and clears them either way.
void set_kernel_events(hipEvent_t start, hipEvent_t stop);
bool take_kernel_events_used();

// Kernel launchers (pcs_kernels.hip).  All are asynchronous on `s`.
enum TileMode : int {
    kModeHash = 0,    // fingerprint the buffer's runs
    kModePack = 1,    // ... and store every chunk to its snapshot slot (checkpoint)
    kModeDiff = 2,    // ... and mark chunks new or changed against the parent (incremental):
                      // bit c of the group's 64-bit mask (an 8-chunk sub-tile writes its
                      // byte of it)
    kModeVerify = 3,  // copy snapshot slots to the buffer's runs (restore), fingerprint
                      // the restored bytes and mark chunks whose fingerprint differs
                      // from the one stored at checkpoint time
};
hipError_t launch_group_map(const JobBuf *bufs, const Run *runs, uint32_t nbuf, uint64_t ngroups, GroupRef *map,
                            hipStream_t s);
// The device a tile launch runs on: its CU count and the rate of its constant
// real-time counter (kHz); zeros: unknown.
struct TileDevice {
    uint32_t cus;
    uint32_t wall_khz;
};
// First-round stagger of whole-group pack and verify jobs of
// kStaggerMinRounds..kStaggerMaxRounds rounds (one workgroup per CU): the
// first round's workgroups start 0..kStaggerPhases-1 phases of
// kStaggerPhaseNs apart (k_hash, stagger_start).  Measured on MI355X (pack +
// fingerprint, one process, against no stagger): 128 MiB -8.4%, 256 MiB
// -13%, 384 MiB -3.5%, 512 MiB -7.3%, the 512 MiB KV ring window -6.8%
// (verified restore -5.5%), 640 MiB +2.0%, 768 MiB +0.2%, 1 GiB +1.6%;
// one-round jobs only lose.
struct Stagger {
    uint32_t first_round;  // workgroups of the first round (0: no stagger)
    uint32_t ticks;        // real-time counter ticks per phase
};
constexpr uint32_t kStaggerPhases = 8, kStaggerMinRounds = 2, kStaggerMaxRounds = 9;
constexpr uint32_t kStaggerPhaseNs = 2000;
constexpr uint32_t kStaggerMaxSpins = 4096;  // bound of a wait (about 0.5 ms) whatever the counter does
template <class Tab>
hipError_t launch_tile(const Tab &tab, uint64_t ngroups, int mode, uint64_t *nodes, uint64_t *flag_mask,
                       uint64_t arena_base, hipStream_t s, uint32_t tiles_per_group = 1,
                       TileDevice dev = TileDevice{0, 0});
// A plain pack of a job within the write-back bound (kPackWriteBackMaxRounds
// rounds of `cus` workgroups) stores write-back, other copies nontemporal
// (cus 0: nontemporal).
template <class Tab>
hipError_t launch_copy(const Tab &tab, uint64_t ngroups, bool pack, uint64_t arena_base, hipStream_t s,
                       uint32_t cus = 0);
// Where the stored chunks of an incremental checkpoint go.  Slot s is the
// 4096 bytes ending s*4096 below the call's payload top (an arena offset).
// The scan that totals the stored chunks takes the top from *bump (or from
// `reset`, nonzero when the call starts a new segment of the arena), writes
// the top lowered by the slots it places to *bump_out (the other of two
// words, so that every workgroup of the launch may still read *bump; the
// next call reads *bump_out), and the top to *top_out, which the copy
// kernels of separate launches read; with bump null it places nothing (the
// host writes *top_out once it has allocated the slots).  host: two mapped
// pinned words that receive the stored-chunk count and the top.
struct SlotBump {
    uint64_t *bump;
    uint64_t *bump_out;
    uint64_t reset;
    uint64_t *top_out;
    uint64_t *host;
};
// Slot assignment + dirty copy of an incremental checkpoint in one launch
// (from the scanned per-group offsets and the dirty masks); writes the whole
// new manifest.
template <class Tab>
hipError_t launch_place_dirty(const Tab &tab, uint64_t ngroups, const uint64_t *dirty_mask, const uint64_t *offsets,
                              const uint64_t *top_word, uint64_t arena_base, hipStream_t s);
template <class Tab>
hipError_t launch_classify(const Tab &tab, uint64_t ngroups, const uint64_t *hashes, uint32_t K, uint64_t total,
                           uint64_t *bitmap, hipStream_t s);
template <class Tab>
hipError_t launch_labels(const Tab &tab, const uint64_t *bitmap, uint8_t *labels, hipStream_t s);
// Classification and labels of a small job (tables in the kernel arguments,
// at most kClassifyFusedGroups groups) in one single-workgroup launch.
constexpr uint64_t kClassifyFusedGroups = 1024;
hipError_t launch_classify_small(const ArgTables &tab, uint64_t ngroups, const uint64_t *hashes, uint32_t K,
                                 uint64_t total, uint64_t *bitmap, uint8_t *labels, hipStream_t s);
// Per-list Merkle reductions (one workgroup per list, or one for all the
// lists of a small job).  pre: every buffer list of more than
// kMerkleLdsValues values had its first level reduced by
// launch_merkle_blocks (into scratch_a at the list's offset).
hipError_t launch_merkle(const MerkleList *lists, uint32_t nlists, const uint64_t *in,
                         uint64_t *scratch_a, uint64_t *scratch_b, uint64_t *roots_out,
                         uint64_t max_count, bool pre, hipStream_t s);
hipError_t launch_merkle_small(const ArgLists &lists, const uint64_t *in, uint64_t *scratch_a,
                               uint64_t *scratch_b, bool pre, hipStream_t s);
hipError_t launch_merkle_blocks(const LongLists &lists, const uint64_t *in, uint64_t *scratch_a, hipStream_t s);
// Exclusive scan of the set-bit counts of per-group dirty masks (offsets
// and total), then the placement of the slots (SlotBump).
hipError_t launch_scan(const uint64_t *dirty_mask, uint64_t n, uint64_t *offsets, uint64_t *total,
                       const SlotBump &bump, hipStream_t s);
constexpr uint64_t kScanCompactMaxGroups = 4096;
// Small incremental jobs (tables in the kernel arguments, at most
// kScanCompactMaxGroups groups), after the fingerprint + diff tiles: one
// launch reduces the Merkle lists, scans the dirty masks (total also to
// *total and the pinned host words), places the slots and copies the dirty
// chunks.  bump.bump and bump.bump_out must differ.
hipError_t launch_merkle_scan_place(const ArgLists &lists, const uint64_t *nodes, uint64_t *scratch_a,
                                    uint64_t *scratch_b, const ArgTables &tab, uint64_t ngroups,
                                    const uint64_t *dirty_mask, const SlotBump &bump, uint64_t *total,
                                    uint64_t arena_base, hipStream_t s);
hipError_t launch_reverse_slots(uint64_t top, uint64_t dst, uint64_t n, hipStream_t s);
// Flips the lowest bit of the byte at device address addr.
hipError_t launch_flip_bit(uint64_t addr, hipStream_t s);
// Bank shrink: kept = the indices of the `keep` best-ranked entries (score
// order of pcs_bank_shrink), in increasing order: a radix select, then
// index-ordered scans.  select_steps(n) launches, step 0 first: one
// single-workgroup launch for small banks, else twelve (scratch: device
// memory of select_scratch_bytes(n) bytes, 256-byte aligned, nothing to
// clear).
uint32_t select_steps(uint32_t n);
uint64_t select_scratch_bytes(uint32_t n);
hipError_t launch_shrink_select(const float *scores, uint32_t n, uint32_t keep, uint32_t *kept, uint64_t scratch,
                                uint32_t step, hipStream_t s);
// Bank shrink moves, all parts: dst entry j <- src entry kept[j], j < keep.
// stage: the pass that copies, for in-place parts (stage != 0), the entries
// a compaction would overwrite before reading them to their staging areas;
// it must run before the place pass (stage false), which writes every
// destination.
hipError_t launch_move_entries(const ShrinkParts &parts, const uint32_t *kept, uint64_t keep, bool stage,
                               hipStream_t s);

}  // namespace pcs

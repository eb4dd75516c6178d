/*
 * pcs.h -- C ABI of libpcs, the GPU byte layer under a Persistent
 * Computational State (PCS) runtime for generative world models.
 *
 * The paper ("Persistent Computational State: A Session-Centric Runtime for
 * Generative World Models") specifies PCS as a contract (Sec. 3, "The
 * contract"): four operations over a session and opaque handles,
 *     c = checkpoint(s),  s' = restore(c),  c' = fork(c),  delete(c),
 * with four invariants: I1 round-trip, I2 durability (a checkpoint is an
 * immutable snapshot, not a live alias), I3 fork independence and
 * I4 snapshot completeness (|checkpoint| = |PCS|).  Which buffers belong to
 * PCS is decided by derivability (Sec. 3, "The partition"): a buffer that
 * re-running the compute does not reproduce must be snapshotted.  Sec. 4
 * measures that by ablation; this library measures it with content
 * fingerprints over K replays (pcs_fingerprint + pcs_classify).
 *
 * Fingerprint definition (the paper names no hash; this is the library's):
 *   - a buffer's logical bytes are cut into 4096-byte chunks counted from its
 *     first logical byte; the last chunk holds only the remaining bytes;
 *   - each chunk's fingerprint is XXH64 with seed 0 of its bytes;
 *   - a buffer's root is the binary Merkle root over its chunk fingerprints:
 *     pairs (2j, 2j+1) of a level form node j of the next level as XXH64
 *     (seed 0) of the 16 bytes left||right, each little-endian; an odd last
 *     node is promoted unchanged; an empty buffer's root is XXH64 of the
 *     empty input (0xEF46DB3751D8E999);
 *   - a session root is the same Merkle tree over the buffer roots in plan
 *     order.
 *
 * Conventions for every entry point:
 *   - Pointers named d_* are device addresses (HIP device memory, or memory
 *     the device can read and write); pointers named h_* are host memory.
 *   - Every call is stream-ordered on the stream given to pcs_ctx_create:
 *     device outputs are valid once that stream reaches the call's end;
 *     handles are valid when the call returns.  Buffers a call reads must not
 *     be modified, and buffers it writes must not be read, by other streams
 *     until then (I2 durability is defined in stream order); every device
 *     buffer a call names stays allocated until then as well.
 *   - Status: PCS_OK (0) or a negative PCS_E_* code.  On an error no handle
 *     was created and pcs_last_error() describes the failure.  Nothing has
 *     been enqueued either, except where an entry point says otherwise: an
 *     image that fails pcs_import's device check (PCS_E_CORRUPT), an
 *     incremental checkpoint that waited for its stored-chunk count and then
 *     found no room for the chunks (PCS_E_NOMEM; its fingerprint outputs were
 *     written), and pcs_discover after its probes ran; each of these has
 *     waited for its work when it returns.  PCS_E_HIP means a HIP call
 *     failed after some work may have been enqueued.
 *   - A context is not thread-safe: use one context per host thread.
 */
#ifndef PCS_H
#define PCS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PCS_OK 0
#define PCS_E_INVAL (-1)   /* bad argument or descriptor                         */
#define PCS_E_NOMEM (-2)   /* the arena cannot hold the request (no eviction)    */
#define PCS_E_HANDLE (-3)  /* unknown or deleted snapshot handle                 */
#define PCS_E_SHAPE (-4)   /* restore target layout differs from the snapshot's  */
#define PCS_E_HIP (-5)     /* a HIP runtime call failed                          */
#define PCS_E_CORRUPT (-6) /* an imported image does not match its fingerprints  */
#define PCS_E_PROBE (-7)   /* the caller's probe reported a failure              */

#define PCS_CHUNK_BYTES 4096u

/* Buffer kinds. */
#define PCS_FLAT 0u  /* nbytes contiguous bytes at ptr                       */
#define PCS_RING 1u  /* a ring-buffered window, see pcs_buf                  */

/* Classification labels (derivability, Sec. 3 "The partition"). */
#define PCS_RECOMPUTABLE 0u
#define PCS_MUST_SNAPSHOT 1u

/* Checkpoint flags. */
#define PCS_CKPT_HASH 1u  /* also fingerprint while copying (one read of the state) */

/* pcs_set_timing modes (see there). */
#define PCS_TIMING_OFF 0
#define PCS_TIMING_EVENTS 1   /* events recorded on the stream around each launch */
#define PCS_TIMING_DISPATCH 2 /* each kernel dispatch's own begin and end        */

typedef struct pcs_ctx pcs_ctx;
typedef uint64_t pcs_snap; /* opaque snapshot handle; 0 is never a valid handle */

/*
 * One candidate buffer of a session's runtime state.
 *
 * PCS_FLAT: `nbytes` bytes starting at `ptr`.  `ptr` must be 16-byte aligned;
 *   nbytes may be any value, including 0, as long as ptr + nbytes stays
 *   below 2^64.  Ring fields are ignored.
 *
 * PCS_RING: the windowed KV context of the paper's addressable-memory model
 *   (Table 1; Sec. 7.11: a context capped by a local window and written at
 *   contiguous positions).  `outer` independent rings (e.g. layers x {K,V});
 *   ring o starts at ptr + o*outer_stride and holds `capacity` rows of
 *   `row_bytes` (a row is one token: heads x head_dim x element size).  The
 *   valid window is `window` rows; logical row t (0 <= t < window) of ring o
 *   lives in physical row (head + t) mod capacity.  The buffer's logical
 *   bytes are ring 0's window rows in order, then ring 1's, and so on:
 *   nbytes = outer * window * row_bytes (pass that value or 0).
 *   Requirements: ptr, row_bytes and outer_stride multiples of 16;
 *   0 <= window <= capacity (an empty window holds no bytes); head <
 *   capacity; outer <= 2^30; outer_stride >= capacity * row_bytes when
 *   outer > 1 (rings do not overlap); ptr + (outer - 1) * outer_stride +
 *   capacity * row_bytes stays below 2^64.
 *
 * Fingerprints and snapshots of a ring cover its logical window, so they do
 * not depend on the head offset: a window restored at a different head
 * fingerprints the same.
 */
typedef struct pcs_buf {
    uint64_t ptr;          /* device address                                  */
    uint64_t nbytes;       /* logical byte count (see above)                  */
    uint32_t kind;         /* PCS_FLAT or PCS_RING                            */
    uint32_t flags;        /* reserved, must be 0                             */
    uint64_t row_bytes;    /* RING: bytes per row                             */
    uint64_t capacity;     /* RING: rows per ring                             */
    uint64_t head;         /* RING: physical row of logical row 0             */
    uint64_t window;       /* RING: valid rows                                */
    uint64_t outer;        /* RING: number of rings                           */
    uint64_t outer_stride; /* RING: bytes from ring o to ring o+1             */
} pcs_buf;

typedef struct pcs_snap_info {
    uint64_t state_bytes;   /* logical bytes a restore writes (I4: sum of plan sizes) */
    uint64_t stored_bytes;  /* payload bytes this snapshot itself holds in the arena  */
    uint64_t total_chunks;  /* chunks over all buffers                                */
    uint64_t dirty_chunks;  /* incremental: chunks stored here; full: total_chunks    */
    uint32_t nbufs;         /* buffers in the plan                                    */
    uint32_t incremental;   /* 1 if taken against a parent                            */
    uint32_t has_hashes;    /* 1 if chunk fingerprints are stored with it             */
    uint32_t reserved;
} pcs_snap_info;

/*
 * Creates a context over a caller-owned device arena.  All snapshot payloads,
 * their stored fingerprints and manifests, and per-call scratch live inside
 * [d_arena, d_arena + arena_bytes); the library never allocates device memory
 * itself.  `hip_stream` is a hipStream_t (NULL = the null stream) on which
 * every call of this context is enqueued.  The arena and the stream are
 * borrowed: the caller keeps them alive until pcs_ctx_destroy returns.
 * d_arena must be 16-byte aligned; the library uses the arena from its first
 * 4096-byte boundary on, in whole 4096-byte units, keeps the first unit for
 * its own bookkeeping words, and PCS_E_INVAL results if fewer than two units
 * remain.  Small pinned host buffers are allocated for descriptor uploads.
 */
int pcs_ctx_create(void *d_arena, uint64_t arena_bytes, void *hip_stream, pcs_ctx **out);

/* Waits for the context's stream, then frees every handle and host resource. */
int pcs_ctx_destroy(pcs_ctx *ctx);

/* Text of the last failure on this context (never NULL; "" if none). */
const char *pcs_last_error(const pcs_ctx *ctx);

/* Host helper: number of 4096-byte chunks of each buffer (h_chunks[i]) and
 * their sum (*total).  Either output may be NULL.  Validates descriptors. */
int pcs_chunk_counts(const pcs_buf *h_bufs, uint32_t n, uint64_t *h_chunks, uint64_t *total);

/*
 * Fingerprints n buffers (chunked XXH64 + Merkle, definition above).
 *   d_chunk_hashes: uint64[total chunks], buffer-major (buffer 0's chunks,
 *                   then buffer 1's ...); may be NULL.
 *   d_roots:        uint64[n], per-buffer Merkle roots; may be NULL.
 *   d_session_root: uint64[1], root over the buffer roots; may be NULL.
 */
int pcs_fingerprint(pcs_ctx *ctx, const pcs_buf *h_bufs, uint32_t n, uint64_t *d_chunk_hashes,
                    uint64_t *d_roots, uint64_t *d_session_root);

/*
 * pcs_fingerprint without allocation, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it).  Same arguments, outputs and stream ordering as pcs_fingerprint, and
 * bit-identical results.  Its descriptor tables, group map and Merkle levels
 * live in a static device array of 16 MiB that every GPU the library runs on
 * holds until the process ends (its address is looked up once per device when
 * the first context on that device is created); the tables of a job of more
 * than 16 buffers or 64 physical runs reach it through a 2 MiB pinned host
 * buffer made by pcs_ctx_create.  The call itself makes no device, pinned or
 * HIP allocation, creates no HIP event (kernel timing skips it) and takes no
 * arena space.
 * Limits: at most 4096 buffers and 65536 physical runs (a ring window is at
 * most two runs per ring), and at most 16 MiB of scratch: about 32 bytes per
 * 64-chunk group (256 KiB of state) plus 160 bytes per buffer and 16 per run
 * (about 120 GiB of state); beyond them PCS_E_INVAL, nothing enqueued.
 * Every call on one GPU shares that GPU's array and it keeps the last call's
 * contents (nothing in it needs clearing: each call writes what it reads):
 * calls that overlap on one GPU (contexts on different streams not ordered
 * against each other) race and give wrong results; calls ordered on one
 * stream do not.
 */
int pcs_fingerprint_noalloc(pcs_ctx *ctx, const pcs_buf *h_bufs, uint32_t n, uint64_t *d_chunk_hashes,
                            uint64_t *d_roots, uint64_t *d_session_root);

/*
 * Cross-replay classification (derivability, Sec. 3 "The partition"; the
 * fingerprint stands in for the Sec. 4 ablation).
 *   d_hashes:  uint64[K][total], replay-major; each replay is laid out like
 *              pcs_fingerprint's d_chunk_hashes for the same plan.
 *   h_chunks:  uint64[n], chunks per buffer (the same in every replay).
 *   d_bitmap:  uint64[sum_b ceil(h_chunks[b]/64)]: each buffer starts on a
 *              fresh word; chunk i of buffer b is bit (i mod 64) of its word
 *              i/64 and is 1 iff its K fingerprints are not all equal.
 *              Unused bits are 0.
 *   d_labels:  uint8[n]: PCS_MUST_SNAPSHOT iff any chunk differs, else
 *              PCS_RECOMPUTABLE.
 * K >= 1 (K = 1 labels everything recomputable).
 */
int pcs_classify(pcs_ctx *ctx, const uint64_t *d_hashes, uint32_t K, const uint64_t *h_chunks,
                 uint32_t n, uint64_t *d_bitmap, uint8_t *d_labels);

/*
 * checkpoint(s) -> c (Sec. 3 contract).  Copies the plan's logical bytes
 * into a new immutable snapshot inside the arena and returns its handle.
 *   parent == 0: full snapshot; component b starts 4096-aligned, in plan
 *     order; padding bytes are zero.  With PCS_CKPT_HASH the chunk
 *     fingerprints are computed from the same read and stored with the
 *     snapshot (needed for it to serve as a parent).
 *   parent != 0: incremental snapshot.  The plan must have the parent's
 *     buffer count and the parent must hold fingerprints.  The plan is
 *     fingerprinted; chunk i of buffer b is stored iff the parent had no
 *     chunk i for b or its fingerprint changed; every other chunk is taken
 *     from the parent chain at restore time.  Stored chunks use one 4096-byte
 *     slot each, in increasing (buffer, chunk) order.  Fingerprints are
 *     always stored (flags are ignored).  The call normally reserves one slot
 *     per chunk and returns the unused part to the arena once the stream has
 *     produced the stored-chunk count; if the arena cannot hold that
 *     reservation it first waits for earlier incremental checkpoints (oldest
 *     first) until their unused reservations are returned, then for its own
 *     count and allocates exactly, and if even
 *     that fails it returns PCS_E_NOMEM after its fingerprint outputs were
 *     written.
 *   d_chunk_hashes, d_roots, d_session_root: optional copies of the
 *     fingerprints, laid out as in pcs_fingerprint (need PCS_CKPT_HASH or a
 *     parent; otherwise pass NULL).
 * The snapshot shares no bytes with the plan buffers (I2): later writes to
 * them do not change it.
 */
int pcs_checkpoint(pcs_ctx *ctx, const pcs_buf *h_plan, uint32_t n, pcs_snap parent, uint32_t flags,
                   uint64_t *d_chunk_hashes, uint64_t *d_roots, uint64_t *d_session_root,
                   pcs_snap *out);

/*
 * Full checkpoints of `sessions` sessions in one launch (batched suspend).
 * The paper's unit of state is the session (Sec. 5, "Unit = session"), and
 * its GPU is time-multiplexed: one session holds the model while every other
 * one is suspended as PCS (Sec. 5, "Structure"; Sec. 7.2 measures up to
 * 1,024 resident sessions).  Suspending many sessions at once is therefore
 * `sessions` independent checkpoint(s) -> c calls of the Sec. 3 contract,
 * each with its own handle and the same I2/I4 guarantees; batching them only
 * shares one launch.
 * Session s's plan is h_plans[off_s .. off_s + h_nbufs[s]) with
 * off_s = sum of the earlier h_nbufs.  Output arrays concatenate the
 * sessions in order (chunk hashes and roots as in pcs_fingerprint;
 * d_session_roots is uint64[sessions]).  h_out receives one handle per
 * session.  Either all snapshots are created or none.
 */
int pcs_checkpoint_batch(pcs_ctx *ctx, const pcs_buf *h_plans, const uint32_t *h_nbufs,
                         uint32_t sessions, uint32_t flags, uint64_t *d_chunk_hashes,
                         uint64_t *d_roots, uint64_t *d_session_roots, pcs_snap *h_out);

/*
 * restore(c) -> s' (Sec. 3 contract, I1).  Writes the snapshot's logical
 * bytes into the n destination buffers.  dst[b] must have snapshot buffer
 * b's logical size; a ring destination must have the same row_bytes, window
 * and outer (its capacity, head and outer_stride may differ, so a window can
 * be restored at a new head).  Only window rows are written.  Destinations
 * must not overlap each other.  Returns PCS_E_SHAPE on a layout mismatch.
 * Restores copy out of the snapshot, so two restores of one snapshot (or of
 * a fork) are independent (I3).  A restore of at most 16 buffers and 64
 * physical runs carries its tables in the kernel arguments and takes no
 * arena space; a larger one uploads them into arena scratch and returns
 * PCS_E_NOMEM if the arena cannot hold that.
 */
int pcs_restore(pcs_ctx *ctx, pcs_snap snap, const pcs_buf *h_dst, uint32_t n);

/*
 * Verified restore: restore(c) as above, fingerprinting every restored chunk
 * from the same read and comparing it with the fingerprint stored at
 * checkpoint time (the snapshot must hold fingerprints).  Detects a snapshot
 * whose bytes changed after it was taken (I2: a snapshot is immutable).
 *   d_bad_bitmap: uint64 words laid out like pcs_classify's bitmap (each
 *                 buffer on fresh words, chunk i = bit i mod 64 of word i/64):
 *                 1 = the restored chunk's fingerprint differs.  Required
 *                 unless the snapshot has no chunks.
 *   d_bad_labels: optional uint8[n]: 1 iff any chunk of that buffer differs.
 * The bytes are restored whether or not they verify.
 */
int pcs_restore_verify(pcs_ctx *ctx, pcs_snap snap, const pcs_buf *h_dst, uint32_t n, uint64_t *d_bad_bitmap,
                       uint8_t *d_bad_labels);

/* Resumes m suspended sessions in one launch: m independent restore(c) -> s'
 * calls of the Sec. 3 contract (I1 each, I3 between them), batched for the
 * time-multiplexed GPU of Sec. 5 ("Structure").  Snapshot j goes to
 * h_dsts[off_j .. off_j + h_nbufs[j]) with off_j = sum of the earlier
 * h_nbufs; each destination set follows pcs_restore's rules.  Everything is
 * validated first: on an error nothing is enqueued. */
int pcs_restore_batch(pcs_ctx *ctx, const pcs_snap *h_snaps, uint32_t m, const pcs_buf *h_dsts,
                      const uint32_t *h_nbufs);

/* fork(c) -> c' (Sec. 3 contract, I3): a new handle on the same immutable
 * snapshot.  No device work. */
int pcs_fork(pcs_ctx *ctx, pcs_snap snap, pcs_snap *out);

/* delete(c) (Sec. 3 contract): drops one handle.  Arena space is released
 * when no handle and no incremental child needs it any more. */
int pcs_delete(pcs_ctx *ctx, pcs_snap snap);

/* Sizes and flags of a snapshot (I4 accounting).  May wait on the stream for
 * an incremental snapshot's stored-chunk count. */
int pcs_snapshot_info(pcs_ctx *ctx, pcs_snap snap, pcs_snap_info *out);

/* Copies the payload this snapshot holds (stored_bytes of pcs_snap_info) to
 * device memory d_dst of capacity `cap` bytes, stream-ordered: a full
 * snapshot in its canonical layout, an incremental one as its stored 4096-byte
 * slots in increasing (buffer, chunk) order.  For an incremental snapshot
 * d_dst must be 16-byte aligned. */
int pcs_snapshot_payload(pcs_ctx *ctx, pcs_snap snap, void *d_dst, uint64_t cap);

/* Read-only view of the payload a snapshot holds: its device address and
 * size (stored_bytes), e.g. to stream it to storage without a copy.  A full
 * snapshot is in its canonical layout; an incremental one stores its slots
 * in decreasing address order (slot 0 highest).  The memory belongs to the
 * library, must not be written (snapshots are immutable, I2) and stays valid
 * until the snapshot's last handle is deleted. */
int pcs_snapshot_view(pcs_ctx *ctx, pcs_snap snap, uint64_t *d_payload, uint64_t *bytes);

/* Copies the snapshot's stored chunk fingerprints (buffer-major) to d_dst,
 * which holds `cap` uint64 values.  PCS_E_INVAL if it has none. */
int pcs_snapshot_hashes(pcs_ctx *ctx, pcs_snap snap, uint64_t *d_dst, uint64_t cap);

/*
 * Durable snapshots across a process boundary (I2 in its strong form: a
 * session survives the death of the process that created it; Sec. 7.2
 * "Across a process boundary").
 *
 * pcs_export writes a self-contained image of the snapshot to host memory
 * h_dst (capacity `cap`) and waits for it, also when it returns an error, so
 * no copy into h_dst is in flight when it returns (after an error h_dst may
 * hold part of an image): a header (layout of every buffer,
 * Merkle roots, chunk fingerprints) and the full logical state in the
 * canonical layout, whether the snapshot is full or incremental.  With
 * h_dst == NULL it only reports the size in *written.  Layout (little-endian):
 *   "PCSIMG01"; u32 version 1; u32 nbufs n; u64 chunks T; u64 state bytes;
 *   u64 payload bytes; u64 flags 0; n x {u32 kind, u32 0, u64 nbytes,
 *   u64 row_bytes, u64 window, u64 outer, u64 0}; n buffer roots and the
 *   session root; T chunk fingerprints; zero padding to a 4096-byte boundary;
 *   the payload (components 4096-aligned, zero padded).
 *
 * pcs_import rebuilds a full snapshot (with fingerprints) from such an image
 * of `size` bytes in this context, fingerprints the imported bytes on the
 * device and returns PCS_E_CORRUPT, creating no handle, if any chunk or root
 * differs from the image.  The header is checked on the host before any byte
 * is copied: a wrong magic, version or flags, nonzero reserved fields, a ring
 * whose shape does not give its size, totals that do not add up, sums that
 * overflow 64 bits, or a size other than the one the header implies are
 * PCS_E_CORRUPT too.  It waits for the stream (also on errors, so the image
 * may be freed when it returns).
 */
int pcs_export(pcs_ctx *ctx, pcs_snap snap, void *h_dst, uint64_t cap, uint64_t *written);
int pcs_import(pcs_ctx *ctx, const void *h_src, uint64_t size, pcs_snap *out);

/*
 * Relevance-keyed bank shrink (Sec. 5, "The two semantic decisions the
 * runtime owns": what to evict is decided by relevance to the return, not by
 * recency; Sec. 7.5 and Tables 5-6: every policy prunes a session's bank to
 * the same retained fraction and differs only in which entries it ranks as
 * worth keeping).
 *
 * A bank is n_entries entries held as nparts component arrays (struct of
 * arrays, e.g. latents and poses); part p's entry i is entry_bytes bytes at
 * src + i * entry_bytes.  d_scores holds n_entries float32 relevance scores
 * on the device (4-byte aligned), supplied by the caller (e.g. pose distance to the anchor);
 * LOWER is more relevant.  Scores are ordered totally by their bit pattern:
 * -inf < ... < -0.0 < +0.0 < ... < +inf < every NaN; equal scores rank the
 * lower index first.  The call keeps the `keep` best-ranked entries and
 * writes them, in increasing original index order (a stable compaction), to
 * dst + j * entry_bytes, j = 0..keep-1, for every part.  dst == src shrinks
 * in place (a kept entry whose source is itself a destination goes through
 * arena scratch, the others move directly); otherwise the keep * entry_bytes bytes
 * at dst must not overlap the n_entries * entry_bytes bytes at src.  No
 * part's destination may overlap another part's source or destination.  If
 * d_kept is not NULL it receives the kept indices (keep uint32 values,
 * increasing).  Asynchronous on the context stream; a following incremental
 * checkpoint of the shrunk bank (parent = the bank's last snapshot) stores
 * only the chunks the shrink changed.
 *
 * Selection takes O(n_entries) work (a radix select of the keep-th score,
 * then index-ordered scans): one workgroup up to 32768 entries, else every
 * CU in twelve launches (six streams over the scores).  The moves of all
 * parts share two launches (the staging of in-place sources, then the
 * placement).
 *
 * Limits and errors: n_entries <= 2^32 - 1 and keep <= n_entries, else
 * PCS_E_INVAL; nparts <= 64; entry_bytes > 0; misaligned scores and
 * overlapping ranges as above are PCS_E_INVAL (nothing is moved);
 * PCS_E_NOMEM if the arena cannot hold the scratch (4 bytes per kept entry
 * when d_kept is NULL, up to 530 KB of selection state above 32768 entries,
 * plus keep * entry_bytes for every in-place part that moves).
 */
/*
 * Kept count of a shrink to a retained fraction (Sec. 7.5 holds the fraction
 * at 12%; Table 6 sweeps 0.04-0.50 and lists the frames each keeps of a bank
 * of about 21).  The fraction is the exact rational num/den (a decimal as
 * written: 0.12 = 12/100), never a binary floating-point approximation of
 * it.  *h_keep = the integer nearest to n_entries * num / den, a tie (an exact
 * half) going to the even neighbour, then raised to 1 if it is 0 and the bank
 * is not empty; 0 for an empty bank.  This reproduces Table 6's column
 * (21 entries: 1, 2, 3, 5, 10).  Host only, no context.  PCS_E_INVAL if
 * h_keep is NULL, den is 0 or num > den.
 */
int pcs_keep_count(uint64_t num, uint64_t den, uint64_t n_entries, uint64_t *h_keep);

typedef struct pcs_bank_part {
    uint64_t src;          /* device address of entry 0 */
    uint64_t dst;          /* device address for kept entry 0 (== src: in place) */
    uint64_t entry_bytes;  /* bytes per entry of this part */
} pcs_bank_part;

int pcs_bank_shrink(pcs_ctx *ctx, const pcs_bank_part *h_parts, uint32_t nparts, uint64_t n_entries,
                    const float *d_scores, uint64_t keep, uint32_t *d_kept);

/*
 * A return-consistency distance at chunk granularity: the metric D that
 * Sec. 4's procedure and Sec. 6's conformance test compare against a
 * tolerance, taken bit-exactly (a restore whose continuation returns to the
 * same bytes has D = 0).  The n buffers are fingerprinted (chunked XXH64, as
 * pcs_fingerprint) and each chunk's fingerprint is compared with
 * d_ref_hashes (uint64[total chunks], laid out as pcs_fingerprint's
 * d_chunk_hashes for the same plan, e.g. from an uninterrupted run).
 *   *h_differing: chunks whose fingerprint differs (may be NULL);
 *   *h_distance:  h_differing / total chunks, 0 when there are no chunks
 *                 (may be NULL).
 * The comparison and the count run on the device; the call then waits for
 * the context's stream (the result is a host value).  d_ref_hashes may be
 * NULL only when the buffers hold no chunks.  Takes arena scratch of 16 bytes
 * per 64-chunk group (PCS_E_NOMEM if it cannot).
 */
int pcs_distance(pcs_ctx *ctx, const pcs_buf *h_bufs, uint32_t n, const uint64_t *d_ref_hashes,
                 uint64_t *h_differing, double *h_distance);

/*
 * Discovering PCS by measurement (Sec. 4, procedure FINGERPRINT).  The
 * model's runtime state is k components H = {h_0 .. h_{k-1}} (pcs_buf
 * descriptors of the live session, taken at the anchor of the probe).  The
 * caller supplies the probe: given a snapshot that holds exactly the
 * components whose mask byte is 1 (in component order), it restores them
 * into a fresh session (the other components keep a fresh session's
 * state), runs its leave-and-return trajectory and writes the
 * return-consistency distance D >= 0 of the continuation to *d_out
 * (Sec. 6's conformance metric; e.g. the fraction of output chunks whose
 * fingerprint differs from an uninterrupted run, via pcs_distance).  It returns 0, or nonzero to abort.  The probe must not
 * modify the live components.
 *
 * The call runs:
 *   1. necessity: for each h_i, probe a snapshot of H without h_i; h_i is
 *      necessary iff D > eps;
 *   2. sufficiency: probe a snapshot of exactly the necessary set N; if
 *      D <= eps, PCS = N;
 *   3. redundancy fallback: otherwise add, one at a time, the component
 *      whose addition gives the smallest D (ties: the lowest index) until
 *      D <= eps or every component is in;
 *   4. PCS and Derivable = H \ PCS go to *out.
 * With control >= 0 it then runs Sec. 4's control against necessity tests
 * that pass for the wrong reason: a full snapshot in which component
 * `control` holds a wrong value (the lowest bit of its first byte flipped)
 * is probed, and the control passes iff D > eps.
 *
 * Every snapshot is a full checkpoint of the subset, created before and
 * deleted after its probe; the call waits for nothing itself (the probe may).
 * Errors: k > 64, control >= k, an empty control component, a null probe ->
 * PCS_E_INVAL; a probe returning nonzero or a negative or NaN distance ->
 * PCS_E_PROBE; checkpoint errors as pcs_checkpoint.
 */
#define PCS_DISCOVER_MAX 64u

typedef int (*pcs_probe_fn)(void *user, pcs_snap snap, const uint8_t *h_mask, uint32_t k, double *d_out);

typedef struct pcs_discovery {
    uint8_t pcs[PCS_DISCOVER_MAX];        /* 1: component i is in the returned PCS             */
    uint8_t necessary[PCS_DISCOVER_MAX];  /* 1: step 1 found component i necessary             */
    double d_without[PCS_DISCOVER_MAX];   /* step 1: D with component i left out               */
    uint32_t added[PCS_DISCOVER_MAX];     /* step 3: components added, in order                */
    double d_necessary;                   /* step 2: D with exactly the necessary set          */
    double d_final;                       /* D with the returned PCS                           */
    double d_control;                     /* D of the control (-1 without a control)           */
    uint32_t n_added;                     /* entries of added[]                                */
    uint32_t probes;                      /* probe runs                                        */
    int32_t control_ok;                   /* 1 passed, 0 failed, -1 no control                 */
    int32_t converged;                    /* 1 iff d_final <= eps                              */
} pcs_discovery;

int pcs_discover(pcs_ctx *ctx, const pcs_buf *h_components, uint32_t k, double eps, int32_t control,
                 pcs_probe_fn probe, void *user, pcs_discovery *out);

/* Arena accounting: bytes in use (snapshots, the worst case of incremental
 * checkpoints whose stored-chunk count has not come back yet, and scratch of
 * calls in progress), bytes free (the rest of the arena less the unit the
 * library keeps), largest free block, live handles.  Does not wait. */
int pcs_arena_stats(pcs_ctx *ctx, uint64_t *used, uint64_t *free_bytes, uint64_t *largest_free,
                    uint64_t *live_handles);

/*
 * Kernel timing.  PCS_TIMING_OFF: off.  While on, every kernel launch is
 * timed with a pair of HIP events on the context stream:
 *   PCS_TIMING_EVENTS: events recorded on the stream just before and after
 *     the launch, so a launch's time includes its dispatch latency (a few
 *     microseconds);
 *   PCS_TIMING_DISPATCH: the kernel dispatch's own begin and end timestamps
 *     (what a kernel trace reports).  Measured on MI355X, it made the step
 *     times of the 1024-session batch (11 ms kernels back to back) more
 *     spread; it suits kernels for which the dispatch latency is not small.
 * Any other mode is PCS_E_INVAL.  pcs_kernel_time waits for the stream, then
 * reports the number of launches and their summed duration in milliseconds
 * for the kernel family `name` ("hash", "pack_hash", "pack", "copy",
 * "verify", "merkle", "classify", "incremental", "map", "shrink", "flip")
 * since the last reset, and resets it.
 */
int pcs_set_timing(pcs_ctx *ctx, int mode);
int pcs_kernel_time(pcs_ctx *ctx, const char *name, uint64_t *launches, double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* PCS_H */

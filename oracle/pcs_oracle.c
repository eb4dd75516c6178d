/*
 * pcs_oracle.c -- CPU oracle for the fingerprint-and-checkpoint path of
 * "Persistent Computational State: A Session-Centric Runtime for Generative
 * World Models".
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
 * definition that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It
 * shares no source, header, table or helper with the HIP library, and the
 * HIP library never calls it.
 *
 * What is computed, and where it comes from:
 *   - The paper's contract (Sec. 3, "The contract") is checkpoint / restore /
 *     fork / delete over opaque handles, with invariants I1 round-trip,
 *     I2 durability, I3 fork independence and I4 snapshot completeness.
 *   - The paper decides must-snapshot versus recomputable by derivability
 *     (Sec. 3, "The partition"): a buffer is derivable iff re-running the
 *     compute reproduces it.  The paper measures that with an ablation
 *     (Sec. 4, procedure FINGERPRINT); this library measures it with content
 *     fingerprints taken over K replays: a chunk whose K fingerprints are not
 *     all equal was not reproduced, so its buffer must be snapshotted.
 *   - The paper names no hash.  The content fingerprint here is XXH64 with
 *     seed 0 over 4096-byte chunks, combined per buffer by a binary Merkle
 *     tree whose odd node at any level is promoted unchanged.
 *
 * Every function is written straight from its definition: no blocking, no
 * fusion, no reordering.  All arithmetic is unsigned 64-bit and wraps mod
 * 2^64.  Multi-byte words are read little-endian, byte by byte, so the
 * result does not depend on the host's byte order.
 *
 * Parity pins (tests/test_oracle_*.py): XXH64 against the independent
 * `xxhash` library over many lengths and seeds; the Merkle root against a
 * recursive largest-power-of-two split; the ring window against numpy.roll;
 * classification against direct byte comparison; pack/unpack, incremental
 * chains and fork against brute-force round trips; snapshot sizes against
 * the byte counts the paper prints in Table 1 and Sec. 7.2; the bank
 * shrink's selection against Python's sort with a key built from float
 * semantics and against a rank-counting definition on small inputs, and the
 * keep count against the frames Table 6 lists per retained fraction.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* XXH64, written from the published xxHash specification (XXH64,     */
/* version 0.1.1 of the spec).                                        */
/* ------------------------------------------------------------------ */

static const uint64_t PRIME64_1 = 0x9E3779B185EBCA87ULL;
static const uint64_t PRIME64_2 = 0xC2B2AE3D27D4EB4FULL;
static const uint64_t PRIME64_3 = 0x165667B19E3779F9ULL;
static const uint64_t PRIME64_4 = 0x85EBCA77C2B2AE63ULL;
static const uint64_t PRIME64_5 = 0x27D4EB2F165667C5ULL;

static uint64_t rotl64(uint64_t x, unsigned r) { return (x << r) | (x >> (64 - r)); }

static uint64_t read_le64(const uint8_t *p)
{
    uint64_t v = 0;
    for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];
    return v;
}

static uint32_t read_le32(const uint8_t *p)
{
    uint32_t v = 0;
    for (int i = 3; i >= 0; --i) v = (v << 8) | p[i];
    return v;
}

/* One accumulator step: add the input lane times prime 2, rotate left by
 * 31, multiply by prime 1. */
static uint64_t xxh_round(uint64_t acc, uint64_t lane)
{
    acc = acc + lane * PRIME64_2;
    acc = rotl64(acc, 31);
    acc = acc * PRIME64_1;
    return acc;
}

/* Folds one of the four accumulators back into the converged value. */
static uint64_t xxh_merge(uint64_t acc, uint64_t v)
{
    acc = acc ^ xxh_round(0, v);
    acc = acc * PRIME64_1 + PRIME64_4;
    return acc;
}

uint64_t orc_xxh64(const uint8_t *p, uint64_t len, uint64_t seed)
{
    uint64_t acc;
    uint64_t pos = 0;

    if (len >= 32) {
        /* Four accumulators, each fed one 8-byte lane of every 32-byte
         * stripe. */
        uint64_t v1 = seed + PRIME64_1 + PRIME64_2;
        uint64_t v2 = seed + PRIME64_2;
        uint64_t v3 = seed;
        uint64_t v4 = seed - PRIME64_1;
        while (len - pos >= 32) {
            v1 = xxh_round(v1, read_le64(p + pos + 0));
            v2 = xxh_round(v2, read_le64(p + pos + 8));
            v3 = xxh_round(v3, read_le64(p + pos + 16));
            v4 = xxh_round(v4, read_le64(p + pos + 24));
            pos += 32;
        }
        acc = rotl64(v1, 1) + rotl64(v2, 7) + rotl64(v3, 12) + rotl64(v4, 18);
        acc = xxh_merge(acc, v1);
        acc = xxh_merge(acc, v2);
        acc = xxh_merge(acc, v3);
        acc = xxh_merge(acc, v4);
    } else {
        acc = seed + PRIME64_5;
    }

    acc = acc + len;

    /* The remaining 0..31 bytes: 8-byte lanes, then one 4-byte lane, then
     * single bytes. */
    while (len - pos >= 8) {
        acc = acc ^ xxh_round(0, read_le64(p + pos));
        acc = rotl64(acc, 27) * PRIME64_1 + PRIME64_4;
        pos += 8;
    }
    if (len - pos >= 4) {
        acc = acc ^ ((uint64_t)read_le32(p + pos) * PRIME64_1);
        acc = rotl64(acc, 23) * PRIME64_2 + PRIME64_3;
        pos += 4;
    }
    while (len - pos >= 1) {
        acc = acc ^ ((uint64_t)p[pos] * PRIME64_5);
        acc = rotl64(acc, 11) * PRIME64_1;
        pos += 1;
    }

    /* Avalanche. */
    acc = acc ^ (acc >> 33);
    acc = acc * PRIME64_2;
    acc = acc ^ (acc >> 29);
    acc = acc * PRIME64_3;
    acc = acc ^ (acc >> 32);
    return acc;
}

/* ------------------------------------------------------------------ */
/* Chunked fingerprints.                                              */
/* ------------------------------------------------------------------ */

#define ORC_CHUNK 4096ULL

/* A buffer of n bytes is cut into chunks [4096 i, min(4096 (i+1), n)),
 * counted from the buffer's own first byte; the last chunk holds only the
 * real bytes (no padding).  An empty buffer has no chunks. */
uint64_t orc_chunk_count(uint64_t nbytes)
{
    return (nbytes + ORC_CHUNK - 1) / ORC_CHUNK;
}

void orc_chunk_hashes(const uint8_t *p, uint64_t nbytes, uint64_t *out)
{
    uint64_t n = orc_chunk_count(nbytes);
    for (uint64_t i = 0; i < n; ++i) {
        uint64_t start = i * ORC_CHUNK;
        uint64_t len = nbytes - start < ORC_CHUNK ? nbytes - start : ORC_CHUNK;
        out[i] = orc_xxh64(p + start, len, 0);
    }
}

/* An internal Merkle node is XXH64 (seed 0) of the 16 bytes formed by the
 * left child then the right child, each written little-endian. */
uint64_t orc_node_hash(uint64_t left, uint64_t right)
{
    uint8_t b[16];
    for (int i = 0; i < 8; ++i) {
        b[i] = (uint8_t)(left >> (8 * i));
        b[8 + i] = (uint8_t)(right >> (8 * i));
    }
    return orc_xxh64(b, 16, 0);
}

/* Binary Merkle root, level by level: pairs (2j, 2j+1) of one level become
 * node j of the next; a level of odd length promotes its last node
 * unchanged.  The root is the single node left.  No leaves: the root is the
 * XXH64 of the empty input.  `work` must hold n values; it is overwritten. */
uint64_t orc_merkle_root(const uint64_t *leaves, uint64_t n, uint64_t *work)
{
    if (n == 0) return orc_xxh64((const uint8_t *)"", 0, 0);
    for (uint64_t i = 0; i < n; ++i) work[i] = leaves[i];
    uint64_t m = n;
    while (m > 1) {
        uint64_t next = 0;
        for (uint64_t j = 0; j + 1 < m; j += 2) work[next++] = orc_node_hash(work[j], work[j + 1]);
        if (m % 2 == 1) work[next++] = work[m - 1];
        m = next;
    }
    return work[0];
}

/* ------------------------------------------------------------------ */
/* Ring-buffered window (the windowed KV context of Table 1 and of    */
/* Sec. 7.11: a context capped by a local window, written at          */
/* contiguous positions).                                             */
/* ------------------------------------------------------------------ */

/* `outer` independent rings, ring o starting at byte o*outer_stride; each
 * holds `capacity` rows of `row_bytes`.  Logical row t (0 <= t < window)
 * of ring o is physical row (head + t) mod capacity.  The logical view is
 * ring 0's window rows in order, then ring 1's, and so on. */
void orc_ring_window(const uint8_t *ring, uint64_t outer, uint64_t outer_stride,
                     uint64_t capacity, uint64_t row_bytes, uint64_t head,
                     uint64_t window, uint8_t *out)
{
    uint64_t k = 0;
    for (uint64_t o = 0; o < outer; ++o)
        for (uint64_t t = 0; t < window; ++t) {
            uint64_t phys = (head + t) % capacity;
            memcpy(out + k, ring + o * outer_stride + phys * row_bytes, row_bytes);
            k += row_bytes;
        }
}

/* Inverse placement: writes a logical window into a ring at head `head`.
 * Rows outside the window are left untouched. */
void orc_ring_place(const uint8_t *logical, uint64_t outer, uint64_t outer_stride,
                    uint64_t capacity, uint64_t row_bytes, uint64_t head,
                    uint64_t window, uint8_t *ring)
{
    uint64_t k = 0;
    for (uint64_t o = 0; o < outer; ++o)
        for (uint64_t t = 0; t < window; ++t) {
            uint64_t phys = (head + t) % capacity;
            memcpy(ring + o * outer_stride + phys * row_bytes, logical + k, row_bytes);
            k += row_bytes;
        }
}

/* ------------------------------------------------------------------ */
/* Cross-replay classification (derivability, Sec. 3 "The partition"; */
/* the load-bearing control of Sec. 4).                               */
/* ------------------------------------------------------------------ */

/* `hashes` holds K replays one after another; each replay is the
 * concatenation, buffer by buffer, of that buffer's chunk fingerprints, and
 * buffer b has chunks_per_buf[b] chunks in every replay.
 *
 * Chunk i of buffer b differs iff its K fingerprints are not all equal.
 * Bitmap: each buffer starts on a fresh 64-bit word; chunk i sets bit
 * (i mod 64) of the buffer's word (i / 64); unused bits are 0.
 * Label: 1 (must-snapshot) iff some chunk differs, else 0 (recomputable).
 * Returns the number of bitmap words written. */
uint64_t orc_classify(const uint64_t *hashes, uint32_t K, const uint64_t *chunks_per_buf,
                      uint32_t nbuf, uint64_t *bitmap, uint8_t *labels)
{
    uint64_t total = 0;
    for (uint32_t b = 0; b < nbuf; ++b) total += chunks_per_buf[b];

    uint64_t first_chunk = 0, first_word = 0;
    for (uint32_t b = 0; b < nbuf; ++b) {
        uint64_t nc = chunks_per_buf[b];
        uint64_t nw = (nc + 63) / 64;
        for (uint64_t w = 0; w < nw; ++w) bitmap[first_word + w] = 0;
        labels[b] = 0;
        for (uint64_t i = 0; i < nc; ++i) {
            uint64_t h0 = hashes[first_chunk + i];
            int differs = 0;
            for (uint32_t k = 1; k < K; ++k)
                if (hashes[(uint64_t)k * total + first_chunk + i] != h0) differs = 1;
            if (differs) {
                bitmap[first_word + i / 64] |= 1ULL << (i % 64);
                labels[b] = 1;
            }
        }
        first_chunk += nc;
        first_word += nw;
    }
    return first_word;
}

/* ------------------------------------------------------------------ */
/* Full checkpoint in the canonical layout (contract, Sec. 3; I4).    */
/* ------------------------------------------------------------------ */

/* Component b starts at offsets[b], a multiple of 4096; it occupies its
 * byte count rounded up to 4096, and the padding bytes are zero.  Returns
 * the payload size. */
uint64_t orc_payload_layout(const uint64_t *nbytes, uint32_t nbuf, uint64_t *offsets)
{
    uint64_t off = 0;
    for (uint32_t b = 0; b < nbuf; ++b) {
        offsets[b] = off;
        off += orc_chunk_count(nbytes[b]) * ORC_CHUNK;
    }
    return off;
}

void orc_pack(const uint8_t *const *bufs, const uint64_t *nbytes, uint32_t nbuf,
              const uint64_t *offsets, uint64_t payload_bytes, uint8_t *payload)
{
    memset(payload, 0, payload_bytes);
    for (uint32_t b = 0; b < nbuf; ++b) memcpy(payload + offsets[b], bufs[b], nbytes[b]);
}

void orc_unpack(const uint8_t *payload, const uint64_t *nbytes, uint32_t nbuf,
                const uint64_t *offsets, uint8_t *const *bufs)
{
    for (uint32_t b = 0; b < nbuf; ++b) memcpy(bufs[b], payload + offsets[b], nbytes[b]);
}

/* ------------------------------------------------------------------ */
/* Incremental checkpoint: the dirty set against a parent snapshot.   */
/* ------------------------------------------------------------------ */

/* Chunk i of buffer b is dirty iff the parent had no chunk i for that
 * buffer, or the parent's fingerprint of chunk i differs from the new one.
 * Both fingerprint arrays are buffer-major concatenations.  dirty[] gets
 * one byte per new chunk.  Returns the number of dirty chunks. */
uint64_t orc_dirty(const uint64_t *hashes, const uint64_t *counts,
                   const uint64_t *parent_hashes, const uint64_t *parent_counts,
                   uint32_t nbuf, uint8_t *dirty)
{
    uint64_t base = 0, pbase = 0, ndirty = 0;
    for (uint32_t b = 0; b < nbuf; ++b) {
        for (uint64_t i = 0; i < counts[b]; ++i) {
            int d = (i >= parent_counts[b]) || (hashes[base + i] != parent_hashes[pbase + i]);
            dirty[base + i] = (uint8_t)d;
            ndirty += (uint64_t)d;
        }
        base += counts[b];
        pbase += parent_counts[b];
    }
    return ndirty;
}

/* ------------------------------------------------------------------ */
/* Relevance-keyed bank shrink (Sec. 5: what to evict is decided by   */
/* relevance to the return, not recency; Sec. 7.5 and Tables 5-6: a   */
/* shrink keeps a fixed fraction of a session's bank entries and the  */
/* policies differ only in which entries they rank as worth keeping). */
/* ------------------------------------------------------------------ */

/* The library's ranking of caller-supplied scores (lower = more relevant):
 * numeric order, -0.0 before +0.0, every NaN after +inf, and among equal
 * scores the lower index first.  Returns 1 iff entry (a, ia) ranks before
 * entry (b, ib). */
static int ranks_before(float a, uint32_t ia, float b, uint32_t ib)
{
    const int na = isnan(a) != 0, nb = isnan(b) != 0;
    if (na || nb) {
        if (na && nb) return ia < ib;
        return nb;  /* a is a number, b is NaN */
    }
    if (a < b) return 1;
    if (a > b) return 0;
    {
        const int sa = signbit(a) != 0, sb = signbit(b) != 0;
        if (sa != sb) return sa;  /* -0.0 before +0.0 */
    }
    return ia < ib;
}

static const float *g_rank_scores; /* qsort has no context argument */

static int cmp_rank(const void *x, const void *y)
{
    const uint32_t i = *(const uint32_t *)x, j = *(const uint32_t *)y;
    if (i == j) return 0;
    return ranks_before(g_rank_scores[i], i, g_rank_scores[j], j) ? -1 : 1;
}

static int cmp_index(const void *x, const void *y)
{
    const uint32_t i = *(const uint32_t *)x, j = *(const uint32_t *)y;
    return (i > j) - (i < j);
}

/* kept[0..keep) = the `keep` best-ranked of n entries, in increasing index
 * order (the order the shrunk bank holds them in).  Returns 0, or -1 if
 * keep > n or memory runs out. */
int orc_bank_select(const float *scores, uint32_t n, uint32_t keep, uint32_t *kept)
{
    uint32_t *order;
    if (keep > n) return -1;
    if (n == 0) return 0;
    order = (uint32_t *)malloc(sizeof(uint32_t) * n);
    if (!order) return -1;
    for (uint32_t i = 0; i < n; ++i) order[i] = i;
    g_rank_scores = scores;
    qsort(order, n, sizeof(uint32_t), cmp_rank);
    memcpy(kept, order, sizeof(uint32_t) * keep);
    qsort(kept, keep, sizeof(uint32_t), cmp_index);
    free(order);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random      */
/* numbers: as easy as 1, 2, 3", SC'11): the counter-based generator   */
/* the mock world model of the discovery procedure (Sec. 4) draws from */
/* (the paper's RNG state is a Philox key and counter, Table 1).       */
/* ------------------------------------------------------------------ */

/* One block: 10 rounds over a 4 x 32-bit counter with a 2 x 32-bit key.
 * A round multiplies counter words 0 and 2 by the two Philox constants
 * into 64-bit products, and mixes the high halves with the other words and
 * the key; the key is bumped by the two Weyl constants between rounds. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

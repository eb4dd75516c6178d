/*
 * A client of libpcs written against the C ABI alone (include/pcs.h plus the
 * HIP runtime's allocation and copy calls): no Python, no torch.  It builds
 * a session of two buffers (a flat buffer with a ragged size and a wrapped
 * ring window), fingerprints it, checkpoints it with fingerprints, forks the
 * snapshot, overwrites the session, restores the fork into it (the ring at
 * a new head) and exports the snapshot to a host image.
 *
 * Then it rewrites chunk 1 of the flat buffer, takes an incremental
 * checkpoint against the first snapshot, classifies the two fingerprint
 * passes (K = 2), imports the exported image and restores from it, and
 * restores the incremental snapshot.
 *
 * Prints, one per line: "hash <i> <hex>" for every chunk fingerprint,
 * "root <b> <hex>", "session <hex>", "restored <0|1>" (1 when every logical
 * byte came back), "image <bytes>", "dirty <chunks stored by the
 * incremental snapshot>", "bitmap <word> <hex>", "label <b> <0|1>",
 * "imported_restored <0|1>" and "incremental_restored <0|1>"; exits 0 when
 * every call succeeded.
 * tests/test_gpu_c_client.py builds it, runs it and checks the fingerprints
 * against the oracle.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "pcs.h"

#define FLAT_BYTES (3 * 4096 + 777)
#define OUTER 2u
#define CAPACITY 16u
#define ROW 256u
#define HEAD 11u
#define WINDOW 12u
#define NEW_HEAD 3u
#define RING_BYTES (OUTER * CAPACITY * ROW)

static uint8_t pattern(uint32_t buf, uint64_t i)
{
    return (uint8_t)((i * 131u + buf * 17u + (i >> 8)) & 0xFFu);
}

#define HIP_OK(x)                                                             \
    do {                                                                      \
        hipError_t e_ = (x);                                                  \
        if (e_ != hipSuccess) {                                               \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));           \
            return 1;                                                         \
        }                                                                     \
    } while (0)

#define PCS_OK_(ctx, x)                                                       \
    do {                                                                      \
        int s_ = (x);                                                         \
        if (s_ != PCS_OK) {                                                   \
            fprintf(stderr, "%s: %d %s\n", #x, s_, pcs_last_error(ctx));      \
            return 1;                                                         \
        }                                                                     \
    } while (0)

static pcs_buf ring_desc(void *p, uint64_t head)
{
    pcs_buf b;
    memset(&b, 0, sizeof b);
    b.ptr = (uint64_t)(uintptr_t)p;
    b.kind = PCS_RING;
    b.row_bytes = ROW;
    b.capacity = CAPACITY;
    b.head = head;
    b.window = WINDOW;
    b.outer = OUTER;
    b.outer_stride = CAPACITY * ROW;
    return b;
}

int main(void)
{
    uint8_t *h_flat = malloc(FLAT_BYTES), *h_ring = malloc(RING_BYTES), *h_back = malloc(RING_BYTES);
    if (!h_flat || !h_ring || !h_back) return 1;
    for (uint64_t i = 0; i < FLAT_BYTES; ++i) h_flat[i] = pattern(0, i);
    for (uint64_t i = 0; i < RING_BYTES; ++i) h_ring[i] = pattern(1, i);

    void *d_arena = NULL, *d_flat = NULL, *d_ring = NULL, *d_hashes = NULL, *d_roots = NULL, *d_sroot = NULL;
    const uint64_t arena_bytes = 8u << 20;
    HIP_OK(hipMalloc(&d_arena, arena_bytes));
    HIP_OK(hipMalloc(&d_flat, FLAT_BYTES));
    HIP_OK(hipMalloc(&d_ring, RING_BYTES));
    HIP_OK(hipMemcpy(d_flat, h_flat, FLAT_BYTES, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_ring, h_ring, RING_BYTES, hipMemcpyHostToDevice));

    pcs_buf plan[2];
    memset(&plan[0], 0, sizeof plan[0]);
    plan[0].ptr = (uint64_t)(uintptr_t)d_flat;
    plan[0].nbytes = FLAT_BYTES;
    plan[0].kind = PCS_FLAT;
    plan[1] = ring_desc(d_ring, HEAD);

    uint64_t chunks[2], total = 0;
    if (pcs_chunk_counts(plan, 2, chunks, &total) != PCS_OK) return 1;
    HIP_OK(hipMalloc(&d_hashes, 8 * total));
    HIP_OK(hipMalloc(&d_roots, 16));
    HIP_OK(hipMalloc(&d_sroot, 8));

    pcs_ctx *ctx = NULL;
    if (pcs_ctx_create(d_arena, arena_bytes, NULL, &ctx) != PCS_OK) return 1;
    PCS_OK_(ctx, pcs_fingerprint(ctx, plan, 2, d_hashes, d_roots, d_sroot));

    pcs_snap snap = 0, fork = 0;
    PCS_OK_(ctx, pcs_checkpoint(ctx, plan, 2, 0, PCS_CKPT_HASH, NULL, NULL, NULL, &snap));
    PCS_OK_(ctx, pcs_fork(ctx, snap, &fork));

    /* Overwrite the session, then restore the fork into it, the ring at a new head. */
    HIP_OK(hipMemset(d_flat, 0, FLAT_BYTES));
    HIP_OK(hipMemset(d_ring, 0, RING_BYTES));
    pcs_buf dst[2] = {plan[0], ring_desc(d_ring, NEW_HEAD)};
    PCS_OK_(ctx, pcs_restore(ctx, fork, dst, 2));
    HIP_OK(hipDeviceSynchronize());

    int ok = 1;
    uint8_t *h_flat_back = malloc(FLAT_BYTES);
    if (!h_flat_back) return 1;
    HIP_OK(hipMemcpy(h_flat_back, d_flat, FLAT_BYTES, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_back, d_ring, RING_BYTES, hipMemcpyDeviceToHost));
    if (memcmp(h_flat_back, h_flat, FLAT_BYTES) != 0) ok = 0;
    for (uint32_t o = 0; o < OUTER; ++o)
        for (uint32_t t = 0; t < WINDOW; ++t) {
            const uint8_t *want = h_ring + o * CAPACITY * ROW + ((HEAD + t) % CAPACITY) * ROW;
            const uint8_t *got = h_back + o * CAPACITY * ROW + ((NEW_HEAD + t) % CAPACITY) * ROW;
            if (memcmp(want, got, ROW) != 0) ok = 0;
        }

    uint64_t image_bytes = 0;
    PCS_OK_(ctx, pcs_export(ctx, snap, NULL, 0, &image_bytes));
    void *image = malloc(image_bytes);
    if (!image) return 1;
    PCS_OK_(ctx, pcs_export(ctx, snap, image, image_bytes, &image_bytes));

    /* Incremental checkpoint after rewriting chunk 1 of the flat buffer;
     * classification of the two fingerprint passes (K = 2); import of the
     * exported image and a restore from it; a restore of the incremental
     * snapshot. */
    uint8_t *h_flat2 = malloc(FLAT_BYTES), *h_chk = malloc(RING_BYTES);
    void *d_k2 = NULL, *d_bitmap = NULL, *d_labels = NULL, *d_flat3 = NULL, *d_ring3 = NULL;
    if (!h_flat2 || !h_chk) return 1;
    memcpy(h_flat2, h_flat, FLAT_BYTES);
    for (uint64_t i = 4096; i < 8192; ++i) h_flat2[i] ^= 0x5A;
    HIP_OK(hipMemcpy(d_flat, h_flat2, FLAT_BYTES, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_ring, h_ring, RING_BYTES, hipMemcpyHostToDevice));
    HIP_OK(hipMalloc(&d_k2, 16 * total));
    HIP_OK(hipMemcpy(d_k2, d_hashes, 8 * total, hipMemcpyDeviceToDevice));
    pcs_snap inc = 0, imp = 0;
    PCS_OK_(ctx, pcs_checkpoint(ctx, plan, 2, snap, 0, (uint64_t *)d_k2 + total, NULL, NULL, &inc));
    pcs_snap_info inf;
    PCS_OK_(ctx, pcs_snapshot_info(ctx, inc, &inf));
    const uint64_t words = (chunks[0] + 63) / 64 + (chunks[1] + 63) / 64;
    HIP_OK(hipMalloc(&d_bitmap, 8 * words));
    HIP_OK(hipMalloc(&d_labels, 2));
    PCS_OK_(ctx, pcs_classify(ctx, (const uint64_t *)d_k2, 2, chunks, 2, (uint64_t *)d_bitmap, (uint8_t *)d_labels));
    PCS_OK_(ctx, pcs_import(ctx, image, image_bytes, &imp));
    HIP_OK(hipMalloc(&d_flat3, FLAT_BYTES));
    HIP_OK(hipMalloc(&d_ring3, RING_BYTES));
    pcs_buf dst3[2] = {plan[0], ring_desc(d_ring3, NEW_HEAD)};
    dst3[0].ptr = (uint64_t)(uintptr_t)d_flat3;
    PCS_OK_(ctx, pcs_restore(ctx, imp, dst3, 2));
    HIP_OK(hipDeviceSynchronize());
    int imported_ok = 1;
    HIP_OK(hipMemcpy(h_flat_back, d_flat3, FLAT_BYTES, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_chk, d_ring3, RING_BYTES, hipMemcpyDeviceToHost));
    if (memcmp(h_flat_back, h_flat, FLAT_BYTES) != 0) imported_ok = 0;
    for (uint32_t o = 0; o < OUTER; ++o)
        for (uint32_t t = 0; t < WINDOW; ++t) {
            const uint8_t *want = h_ring + o * CAPACITY * ROW + ((HEAD + t) % CAPACITY) * ROW;
            const uint8_t *got = h_chk + o * CAPACITY * ROW + ((NEW_HEAD + t) % CAPACITY) * ROW;
            if (memcmp(want, got, ROW) != 0) imported_ok = 0;
        }
    PCS_OK_(ctx, pcs_restore(ctx, inc, dst3, 2));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(h_flat_back, d_flat3, FLAT_BYTES, hipMemcpyDeviceToHost));
    const int incremental_ok = memcmp(h_flat_back, h_flat2, FLAT_BYTES) == 0;
    uint64_t h_bitmap[4] = {0, 0, 0, 0};
    uint8_t h_labels[2] = {7, 7};
    if (words > 4) return 1;
    HIP_OK(hipMemcpy(h_bitmap, d_bitmap, 8 * words, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_labels, d_labels, 2, hipMemcpyDeviceToHost));
    printf("dirty %llu\n", (unsigned long long)inf.dirty_chunks);
    for (uint64_t w = 0; w < words; ++w) printf("bitmap %llu %016llx\n", (unsigned long long)w, (unsigned long long)h_bitmap[w]);
    printf("label 0 %d\nlabel 1 %d\n", h_labels[0], h_labels[1]);
    printf("imported_restored %d\nincremental_restored %d\n", imported_ok, incremental_ok);

    /* Return-consistency distance of the current bytes (chunk 1 of the flat
     * buffer rewritten) against the first fingerprints. */
    uint64_t differing = 0;
    double distance = -1.0;
    PCS_OK_(ctx, pcs_distance(ctx, plan, 2, (const uint64_t *)d_hashes, &differing, &distance));
    printf("differing %llu\ndistance %.17g\n", (unsigned long long)differing, distance);

    /* Relevance-keyed shrink of a 21-entry bank to 12%: latents in place,
     * poses into another buffer. */
    enum { BANK = 21, LAT = 40, POSE = 12 };
    uint64_t keep = 0;
    if (pcs_keep_count(12, 100, BANK, &keep) != PCS_OK || keep == 0 || keep > BANK) return 1;
    uint8_t h_lat[BANK * LAT], h_pose[BANK * POSE];
    float h_scores[BANK];
    for (int i = 0; i < BANK; ++i) {
        for (int j = 0; j < LAT; ++j) h_lat[i * LAT + j] = (uint8_t)(i * 13 + j * 7);
        for (int j = 0; j < POSE; ++j) h_pose[i * POSE + j] = (uint8_t)(i * 29 + j * 3 + 5);
        h_scores[i] = (float)((i * 37) % 11) - 5.0f;
    }
    void *d_lat, *d_pose, *d_pose_out, *d_scores, *d_kept;
    HIP_OK(hipMalloc(&d_lat, sizeof h_lat));
    HIP_OK(hipMalloc(&d_pose, sizeof h_pose));
    HIP_OK(hipMalloc(&d_pose_out, keep * POSE));
    HIP_OK(hipMalloc(&d_scores, sizeof h_scores));
    HIP_OK(hipMalloc(&d_kept, 4 * keep));
    HIP_OK(hipMemcpy(d_lat, h_lat, sizeof h_lat, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_pose, h_pose, sizeof h_pose, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_scores, h_scores, sizeof h_scores, hipMemcpyHostToDevice));
    const pcs_bank_part parts[2] = {
        {.src = (uint64_t)(uintptr_t)d_lat, .dst = (uint64_t)(uintptr_t)d_lat, .entry_bytes = LAT},
        {.src = (uint64_t)(uintptr_t)d_pose, .dst = (uint64_t)(uintptr_t)d_pose_out, .entry_bytes = POSE},
    };
    PCS_OK_(ctx, pcs_bank_shrink(ctx, parts, 2, BANK, (const float *)d_scores, keep, (uint32_t *)d_kept));
    HIP_OK(hipDeviceSynchronize());
    uint32_t h_kept[BANK];
    HIP_OK(hipMemcpy(h_kept, d_kept, 4 * keep, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_lat, d_lat, keep * LAT, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_pose, d_pose_out, keep * POSE, hipMemcpyDeviceToHost));
    printf("keep %llu\n", (unsigned long long)keep);
    for (uint64_t j = 0; j < keep; ++j) printf("kept %llu %u\n", (unsigned long long)j, h_kept[j]);
    printf("shrunk_lat ");
    for (uint64_t b = 0; b < keep * LAT; ++b) printf("%02x", h_lat[b]);
    printf("\nshrunk_pose ");
    for (uint64_t b = 0; b < keep * POSE; ++b) printf("%02x", h_pose[b]);
    printf("\n");
    (void)hipFree(d_lat);
    (void)hipFree(d_pose);
    (void)hipFree(d_pose_out);
    (void)hipFree(d_scores);
    (void)hipFree(d_kept);
    PCS_OK_(ctx, pcs_delete(ctx, imp));
    PCS_OK_(ctx, pcs_delete(ctx, inc));
    (void)hipFree(d_k2);
    (void)hipFree(d_bitmap);
    (void)hipFree(d_labels);
    (void)hipFree(d_flat3);
    (void)hipFree(d_ring3);
    free(h_flat2);
    free(h_chk);

    uint64_t *h_hashes = malloc(8 * total), h_roots[2], h_sroot;
    if (!h_hashes) return 1;
    HIP_OK(hipMemcpy(h_hashes, d_hashes, 8 * total, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h_roots, d_roots, 16, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(&h_sroot, d_sroot, 8, hipMemcpyDeviceToHost));
    for (uint64_t i = 0; i < total; ++i) printf("hash %llu %016llx\n", (unsigned long long)i, (unsigned long long)h_hashes[i]);
    for (int b = 0; b < 2; ++b) printf("root %d %016llx\n", b, (unsigned long long)h_roots[b]);
    printf("session %016llx\n", (unsigned long long)h_sroot);
    printf("restored %d\n", ok);
    printf("image %llu\n", (unsigned long long)image_bytes);

    PCS_OK_(ctx, pcs_delete(ctx, fork));
    PCS_OK_(ctx, pcs_delete(ctx, snap));
    PCS_OK_(ctx, pcs_ctx_destroy(ctx));
    free(image);
    free(h_hashes);
    free(h_flat_back);
    free(h_flat);
    free(h_ring);
    free(h_back);
    (void)hipFree(d_hashes);
    (void)hipFree(d_roots);
    (void)hipFree(d_sroot);
    (void)hipFree(d_flat);
    (void)hipFree(d_ring);
    (void)hipFree(d_arena);
    return 0;
}

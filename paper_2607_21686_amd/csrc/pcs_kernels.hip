// pcs_kernels.hip -- gfx950 (CDNA4) kernels of libpcs: chunked XXH64 with a
// Merkle combine, fused pack + fingerprint, scatter restore, incremental
// dirty-chunk packing and cross-replay classification.
//
// Work decomposition shared by every kernel: a job is a table of buffers,
// each cut into 4096-byte chunks, and the chunks of one buffer into aligned
// groups of 64.  One workgroup handles one group; a group-to-buffer map
// (k_group_map) replaces any per-block search.  Groups never straddle
// buffers, so a group's 64 chunk fingerprints reduce to one Merkle node
// inside the workgroup (a promote-odd tree over n leaves splits into aligned
// 64-leaf subtrees), and a group is exactly one word of the classification
// bitmap.
//
// Memory traffic is 16-byte vector loads and stores throughout.  Nothing
// here is a contraction, so no MFMA is used; the hash is 64-bit integer
// multiply work on the vector ALU.
#include "pcs_device.h"

namespace pcs {
namespace {

// XXH64 primes (xxHash specification).
constexpr uint64_t P1 = 0x9E3779B185EBCA87ULL;
constexpr uint64_t P2 = 0xC2B2AE3D27D4EB4FULL;
constexpr uint64_t P3 = 0x165667B19E3779F9ULL;
constexpr uint64_t P4 = 0x85EBCA77C2B2AE63ULL;
constexpr uint64_t P5 = 0x27D4EB2F165667C5ULL;

__device__ __forceinline__ uint64_t umin(uint64_t a, uint64_t b) { return a < b ? a : b; }

// 64-bit rotate left by a constant 0 < r < 32: two v_alignbit_b32.
__device__ __forceinline__ uint64_t rotl(uint64_t x, int r)
{
    const uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
    const uint32_t nhi = __builtin_amdgcn_alignbit(hi, lo, 32 - r);
    const uint32_t nlo = __builtin_amdgcn_alignbit(lo, hi, 32 - r);
    return ((uint64_t)nhi << 32) | nlo;
}

// Accumulator step: add lane * P2, rotate left 31, multiply by P1.
__device__ __forceinline__ uint64_t xround(uint64_t acc, uint64_t lane)
{
    acc += lane * P2;
    acc = rotl(acc, 31);
    return acc * P1;
}

__device__ __forceinline__ uint64_t xmerge(uint64_t acc, uint64_t v)
{
    acc ^= xround(0, v);
    return acc * P1 + P4;
}

__device__ __forceinline__ uint64_t avalanche(uint64_t h)
{
    h ^= h >> 33;
    h *= P2;
    h ^= h >> 29;
    h *= P3;
    h ^= h >> 32;
    return h;
}

// XXH64 (seed 0) of the empty input: the short-input start value, length 0,
// no tail, avalanche.
__device__ __forceinline__ uint64_t empty_hash() { return avalanche(P5); }

// XXH64 (seed 0) of the 16 bytes le64(l) || le64(r): the Merkle node.
__device__ __forceinline__ uint64_t node_hash(uint64_t l, uint64_t r)
{
    uint64_t acc = P5 + 16;
    acc ^= xround(0, l);
    acc = rotl(acc, 27) * P1 + P4;
    acc ^= xround(0, r);
    acc = rotl(acc, 27) * P1 + P4;
    return avalanche(acc);
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src)
{
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, 64);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Promote-odd Merkle reduction of lanes [0, m) of one wavefront (m <= 64,
// wave-uniform).  The result is valid in lane 0.
__device__ uint64_t wave_merkle(uint64_t v, uint32_t m)
{
    const int lane = (int)(threadIdx.x & 63);
    while (m > 1) {
        const uint64_t a = shfl64(v, (2 * lane) & 63);
        const uint64_t b = shfl64(v, (2 * lane + 1) & 63);
        const uint32_t half = m >> 1;
        if ((uint32_t)lane < half)
            v = node_hash(a, b);
        else if ((uint32_t)lane == half && (m & 1))
            v = a;  // lane 2*half = m-1: the odd node is promoted
        m = (m + 1) >> 1;
    }
    return v;
}

// Logical-to-physical cursor over one buffer's runs.  Logical offsets fed to
// cursor_addr must not decrease.
struct Cursor {
    const Run *runs;
    uint32_t idx, last;  // current run, last run of the buffer
    uint64_t run_end;    // logical end of the current run
    uint64_t delta;      // physical address minus logical offset (mod 2^64)
    uint64_t nbytes;
};

__device__ __forceinline__ void cursor_load(Cursor &c)
{
    const Run r = c.runs[c.idx];
    c.delta = r.addr - r.lstart;
    c.run_end = c.idx < c.last ? c.runs[c.idx + 1].lstart : c.nbytes;
}

__device__ __forceinline__ Cursor cursor_seek(const Run *runs, uint32_t begin, uint32_t count,
                                              uint64_t nbytes, uint64_t L)
{
    Cursor c;
    c.runs = runs;
    c.last = begin + count - 1;
    c.nbytes = nbytes;
    uint32_t lo = begin, hi = begin + count;  // largest idx with lstart <= L
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (runs[mid].lstart <= L) lo = mid; else hi = mid;
    }
    c.idx = lo;
    cursor_load(c);
    return c;
}

__device__ __forceinline__ uint64_t cursor_addr(Cursor &c, uint64_t L)
{
    while (L >= c.run_end && c.idx < c.last) {
        ++c.idx;
        cursor_load(c);
    }
    return L + c.delta;
}

// Device addresses arrive as integers; casting them to the global address
// space makes the compiler emit global_* (not flat_*) memory instructions.
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) v4u32 g_v4u32;
typedef __attribute__((address_space(1))) uint64_t g_u64;
typedef __attribute__((address_space(1))) uint32_t g_u32;
typedef __attribute__((address_space(1))) uint8_t g_u8;

__device__ __forceinline__ uint4 load16(uint64_t a)
{
    const v4u32 v = *(const g_v4u32 *)a;
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store16(uint64_t a, uint4 v)
{
    const v4u32 w = {v.x, v.y, v.z, v.w};
    *(g_v4u32 *)a = w;
}

// Bytes [0, n) of a granule from `a` (n < 16), zero above: in-bounds reads only.
__device__ uint4 load_partial(uint64_t a, uint32_t n)
{
    uint32_t w[4] = {0, 0, 0, 0};
    const g_u8 *p = (const g_u8 *)a;
    for (uint32_t k = 0; k < n; ++k) w[k >> 2] |= (uint32_t)p[k] << (8 * (k & 3));
    return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ void store_partial(uint64_t a, uint4 v, uint32_t n)
{
    g_u8 *p = (g_u8 *)a;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    for (uint32_t k = 0; k < n; ++k) p[k] = (uint8_t)(w[k >> 2] >> (8 * (k & 3)));
}

// ---------------------------------------------------------------- group map

__global__ void k_group_map(const JobBuf *__restrict__ bufs, uint32_t nbuf, uint64_t ngroups,
                            uint32_t *__restrict__ map)
{
    const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= ngroups) return;
    uint32_t lo = 0, hi = nbuf;  // largest b with group_begin <= g (empty buffers lose ties)
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (bufs[mid].group_begin <= g) lo = mid; else hi = mid;
    }
    map[g] = lo;
}

// ---------------------------------------------------------------- fingerprint

// One workgroup = one 64-chunk group; two lanes per chunk.  Lane p of a pair
// owns XXH64 accumulators 2p and 2p+1, which read exactly the 16 bytes at
// offset 16p of every 32-byte stripe, so each lane's data arrives in one
// 16-byte load per stripe and no lane exchange is needed until the final
// convergence.  COPY also writes every loaded granule to the chunk's
// snapshot slot (zero-padding a partial last chunk): one read of the state
// both packs and fingerprints it.  DIFF marks chunks that are new or changed
// against the parent's fingerprints and counts them per group.
constexpr int kHashBatch = 8;

template <bool COPY, bool DIFF>
__global__ __launch_bounds__(128) void k_hash(const JobBuf *__restrict__ bufs,
                                              const Run *__restrict__ runs,
                                              const uint32_t *__restrict__ map,
                                              uint64_t *__restrict__ nodes,
                                              uint32_t *__restrict__ dirty_count,
                                              uint64_t *__restrict__ dirty_mask)
{
    __shared__ uint64_t leaves[kGroupChunks];
    __shared__ uint32_t dflag[kGroupChunks];

    const uint64_t G = blockIdx.x;
    const JobBuf &jb = bufs[map[G]];
    const uint32_t t = threadIdx.x, ci = t >> 1, p = t & 1;
    const uint64_t gl = G - jb.group_begin;
    const uint64_t nchunks = jb.nchunks, nbytes = jb.nbytes;
    const uint32_t nv = (uint32_t)umin(kGroupChunks, nchunks - gl * kGroupChunks);
    const uint64_t i = gl * kGroupChunks + ci;

    if (ci < nv) {
        const uint64_t cbase = i * kChunk;
        const uint32_t len = (uint32_t)umin(kChunk, nbytes - cbase);
        const uint32_t nst = len >> 5;
        const uint64_t L0 = cbase + 16 * p;
        Cursor cur = cursor_seek(runs, jb.run_begin, jb.run_count, nbytes, L0);
        const uint64_t dst = COPY ? jb.payload + cbase : 0;

        uint64_t va = p ? 0 : P1 + P2;   // accumulator 2p   (seed 0)
        uint64_t vb = p ? 0 - P1 : P2;   // accumulator 2p+1
        if (len == kChunk && L0 + kChunk - 16 <= cur.run_end) {
            // Whole chunk in one physical run: batches of kHashBatch stripes,
            // the next batch's loads in flight while this one is hashed.
            const uint64_t a0 = L0 + cur.delta;
            const uint64_t d0 = dst + 16 * p;
            uint4 d[kHashBatch], n[kHashBatch];
#pragma unroll
            for (int u = 0; u < kHashBatch; ++u) d[u] = load16(a0 + 32 * u);
            for (uint32_t s = 0; s < kChunk / 32; s += kHashBatch) {
                if (s + kHashBatch < kChunk / 32) {
#pragma unroll
                    for (int u = 0; u < kHashBatch; ++u) n[u] = load16(a0 + 32 * (uint64_t)(s + kHashBatch + u));
                }
#pragma unroll
                for (int u = 0; u < kHashBatch; ++u) {
                    if (COPY) store16(d0 + 32 * (uint64_t)(s + u), d[u]);
                    va = xround(va, ((uint64_t)d[u].y << 32) | d[u].x);
                    vb = xround(vb, ((uint64_t)d[u].w << 32) | d[u].z);
                }
#pragma unroll
                for (int u = 0; u < kHashBatch; ++u) d[u] = n[u];
            }
        } else {
            for (uint32_t s = 0; s < nst; ++s) {
                const uint64_t L = L0 + 32 * (uint64_t)s;
                const uint4 d = load16(cursor_addr(cur, L));
                if (COPY) store16(dst + 32 * (uint64_t)s + 16 * p, d);
                va = xround(va, ((uint64_t)d.y << 32) | d.x);
                vb = xround(vb, ((uint64_t)d.w << 32) | d.z);
            }
        }
        const uint64_t oa = shfl64(va, (int)(t ^ 1) & 63);
        const uint64_t ob = shfl64(vb, (int)(t ^ 1) & 63);

        uint64_t h = 0;
        if (p == 0) {
            uint64_t acc;
            if (len >= 32) {
                acc = rotl(va, 1) + rotl(vb, 7) + rotl(oa, 12) + rotl(ob, 18);
                acc = xmerge(acc, va);
                acc = xmerge(acc, vb);
                acc = xmerge(acc, oa);
                acc = xmerge(acc, ob);
            } else {
                acc = P5;
            }
            acc += len;
            uint32_t pos = nst * 32;
            if (pos < len) {
                // The tail lies in one run: runs are 16-byte granular and
                // only a flat buffer (a single run) has a tail that is not a
                // whole granule.  Naturally aligned, in-bounds loads only.
                uint64_t tp = cursor_addr(cur, cbase + pos);
                for (; len - pos >= 8; pos += 8, tp += 8) {
                    acc ^= xround(0, *(const g_u64 *)tp);
                    acc = rotl(acc, 27) * P1 + P4;
                }
                if (len - pos >= 4) {
                    acc ^= (uint64_t)(*(const g_u32 *)tp) * P1;
                    acc = rotl(acc, 23) * P2 + P3;
                    pos += 4;
                    tp += 4;
                }
                for (; pos < len; ++pos, ++tp) {
                    acc ^= (uint64_t)(*(const g_u8 *)tp) * P5;
                    acc = rotl(acc, 11) * P1;
                }
            }
            h = avalanche(acc);
        }

        if (COPY && len < kChunk) {
            // Tail and zero padding of the last chunk's slot, granule by
            // granule (after the hash tail, so the cursor only moves forward).
            for (uint32_t q = 2 * nst + p; q < kChunk / 16; q += 2) {
                const uint32_t lo = 16 * q;
                uint4 v = make_uint4(0, 0, 0, 0);
                if (lo + 16 <= len) v = load16(cursor_addr(cur, cbase + lo));
                else if (lo < len) v = load_partial(cursor_addr(cur, cbase + lo), len - lo);
                store16(dst + lo, v);
            }
        }

        if (p == 0) {
            if (jb.hash_dst[0]) ((g_u64 *)jb.hash_dst[0])[i] = h;
            if (jb.hash_dst[1]) ((g_u64 *)jb.hash_dst[1])[i] = h;
            leaves[ci] = h;
            if (DIFF) {
                const bool d = i >= jb.parent_chunks ||
                               ((const g_u64 *)jb.parent_hash)[i] != h;
                dflag[ci] = d ? 1u : 0u;
            }
        }
    }
    __syncthreads();
    if (t < 64) {
        const uint64_t v = t < nv ? leaves[t] : 0;
        const uint64_t r = wave_merkle(v, nv);
        if (t == 0) nodes[G] = r;
        if (DIFF) {
            const uint64_t mask = __ballot(t < nv && dflag[t] != 0);
            if (t == 0) {
                dirty_mask[G] = mask;
                dirty_count[G] = (uint32_t)__popcll(mask);
            }
        }
    }
}

// ---------------------------------------------------------------- Merkle lists

// One workgroup per list: promote-odd Merkle root of in[begin, begin+count).
// Aligned 64-value blocks reduce independently (one wavefront each); up to
// two passes through global scratch bring a list to <= 4096 values, then
// the rest happens in LDS.  Each scratch array is read only after it is
// fully written in this launch.
__global__ __launch_bounds__(256) void k_merkle(const MerkleList *__restrict__ lists,
                                                const uint64_t *__restrict__ in,
                                                uint64_t *__restrict__ sa, uint64_t *__restrict__ sb,
                                                uint64_t *__restrict__ roots_out)
{
    __shared__ uint64_t lds[4096];
    __shared__ uint64_t lds2[64];
    const MerkleList Lst = lists[blockIdx.x];
    const uint32_t t = threadIdx.x, wave = t >> 6, lane = t & 63;
    uint64_t m = Lst.count;
    uint64_t root = 0;
    if (m == 0) {
        root = empty_hash();
    } else {
        const uint64_t *src = in + Lst.begin;
        uint64_t *scratch[2] = {sa + Lst.begin, sb + Lst.begin};
        for (int k = 0; k < 2 && m > 4096; ++k) {
            const uint64_t nb = (m + 63) / 64;
            for (uint64_t blk = wave; blk < nb; blk += 4) {
                const uint32_t cnt = (uint32_t)umin(64, m - 64 * blk);
                const uint64_t v = lane < cnt ? src[64 * blk + lane] : 0;
                const uint64_t r = wave_merkle(v, cnt);
                if (lane == 0) scratch[k][blk] = r;
            }
            __syncthreads();
            src = scratch[k];
            m = nb;
        }
        for (uint64_t j = t; j < m; j += 256) lds[j] = src[j];
        __syncthreads();
        const uint64_t *ls = lds;
        if (m > 64) {
            const uint64_t nb = (m + 63) / 64;
            for (uint64_t blk = wave; blk < nb; blk += 4) {
                const uint32_t cnt = (uint32_t)umin(64, m - 64 * blk);
                const uint64_t v = lane < cnt ? lds[64 * blk + lane] : 0;
                const uint64_t r = wave_merkle(v, cnt);
                if (lane == 0) lds2[blk] = r;
            }
            __syncthreads();
            ls = lds2;
            m = nb;
        }
        if (wave == 0) {
            const uint64_t v = lane < m ? ls[lane] : 0;
            root = wave_merkle(v, (uint32_t)m);
        }
    }
    if (t == 0) {
        if (Lst.dst[0]) *(g_u64 *)Lst.dst[0] = root;
        if (Lst.dst[1]) *(g_u64 *)Lst.dst[1] = root;
        if (roots_out) roots_out[blockIdx.x] = root;
    }
}

// ---------------------------------------------------------------- copies

constexpr int kCopyUnroll = 4;

// Pack: one workgroup copies its group's chunks, 256 lanes x 16 bytes = one
// whole 4096-byte chunk per step (fully coalesced on both sides), from the
// buffer's runs into the snapshot slots; a partial last chunk is
// zero-padded to the end of its slot.
__global__ __launch_bounds__(256) void k_pack(const JobBuf *__restrict__ bufs,
                                              const Run *__restrict__ runs,
                                              const uint32_t *__restrict__ map)
{
    const uint64_t G = blockIdx.x;
    const JobBuf &jb = bufs[map[G]];
    const uint64_t gl = G - jb.group_begin;
    const uint64_t c0 = gl * kGroupChunks, nbytes = jb.nbytes;
    const uint32_t nv = (uint32_t)umin(kGroupChunks, jb.nchunks - c0);
    const uint32_t x = threadIdx.x * 16;
    Cursor cur = cursor_seek(runs, jb.run_begin, jb.run_count, nbytes, c0 * kChunk + x);
    for (uint32_t k = 0; k < nv; k += kCopyUnroll) {
        uint4 v[kCopyUnroll];
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u) {
            const uint64_t cb = (c0 + k + u) * kChunk;
            v[u] = make_uint4(0, 0, 0, 0);
            if (k + u < nv) {
                if (cb + x + 16 <= nbytes) v[u] = load16(cursor_addr(cur, cb + x));
                else if (cb + x < nbytes) v[u] = load_partial(cursor_addr(cur, cb + x), (uint32_t)(nbytes - cb - x));
            }
        }
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u)
            if (k + u < nv) store16(jb.payload + (c0 + k + u) * kChunk + x, v[u]);
    }
}

// Restore: snapshot slots (contiguous, or per-chunk through a manifest of
// arena offsets) back into the destination buffer's runs.  Only logical
// bytes are written.
__global__ __launch_bounds__(256) void k_restore(const JobBuf *__restrict__ bufs,
                                                 const Run *__restrict__ runs,
                                                 const uint32_t *__restrict__ map,
                                                 uint64_t arena_base)
{
    const uint64_t G = blockIdx.x;
    const JobBuf &jb = bufs[map[G]];
    const uint64_t gl = G - jb.group_begin;
    const uint64_t c0 = gl * kGroupChunks, nbytes = jb.nbytes;
    const uint32_t nv = (uint32_t)umin(kGroupChunks, jb.nchunks - c0);
    const uint32_t x = threadIdx.x * 16;
    const g_u64 *man = (const g_u64 *)jb.manifest;
    Cursor cur = cursor_seek(runs, jb.run_begin, jb.run_count, nbytes, c0 * kChunk + x);
    for (uint32_t k = 0; k < nv; k += kCopyUnroll) {
        uint4 v[kCopyUnroll];
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u) {
            const uint64_t c = c0 + k + u;
            v[u] = make_uint4(0, 0, 0, 0);
            if (k + u < nv && c * kChunk + x < nbytes) {
                const uint64_t src = man ? arena_base + man[c] : jb.payload + c * kChunk;
                v[u] = load16(src + x);  // slots are whole 4096-byte granules
            }
        }
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u) {
            const uint64_t cb = (c0 + k + u) * kChunk;
            if (k + u < nv) {
                if (cb + x + 16 <= nbytes) store16(cursor_addr(cur, cb + x), v[u]);
                else if (cb + x < nbytes) store_partial(cursor_addr(cur, cb + x), v[u], (uint32_t)(nbytes - cb - x));
            }
        }
    }
}

// ---------------------------------------------------------------- incremental

// Exclusive scan of per-group dirty counts (one workgroup; Hillis-Steele
// over 1024 per-thread partial sums).
__global__ __launch_bounds__(1024) void k_scan(const uint32_t *__restrict__ counts, uint64_t n,
                                               uint64_t *__restrict__ offsets,
                                               uint64_t *__restrict__ total)
{
    __shared__ uint64_t sums[2][1024];
    const uint32_t t = threadIdx.x;
    const uint64_t per = (n + 1023) / 1024;
    const uint64_t s0 = umin(n, t * per), s1 = umin(n, s0 + per);
    uint64_t s = 0;
    for (uint64_t j = s0; j < s1; ++j) s += counts[j];
    int cur = 0;
    sums[0][t] = s;
    __syncthreads();
    for (uint32_t d = 1; d < 1024; d <<= 1) {
        const uint64_t v = sums[cur][t] + (t >= d ? sums[cur][t - d] : 0);
        sums[cur ^ 1][t] = v;
        cur ^= 1;
        __syncthreads();
    }
    uint64_t run = sums[cur][t] - s;  // exclusive prefix of this thread's segment
    for (uint64_t j = s0; j < s1; ++j) {
        offsets[j] = run;
        run += counts[j];
    }
    if (t == 1023) *total = sums[cur][t];
}

// Assigns slots to dirty chunks in (buffer, chunk) order, lists them, and
// writes the new snapshot's manifest: a dirty chunk points at its slot, a
// clean one at wherever the parent holds it.
__global__ __launch_bounds__(64) void k_compact(const JobBuf *__restrict__ bufs,
                                                const uint32_t *__restrict__ map,
                                                const uint64_t *__restrict__ dirty_mask,
                                                const uint64_t *__restrict__ offsets,
                                                uint64_t payload_arena_off,
                                                uint64_t *__restrict__ list)
{
    const uint64_t G = blockIdx.x;
    const uint32_t b = map[G];
    const JobBuf &jb = bufs[b];
    const uint32_t lane = threadIdx.x;
    const uint64_t gl = G - jb.group_begin;
    const uint64_t i = gl * kGroupChunks + lane;
    if (i >= jb.nchunks) return;
    const uint64_t mask = dirty_mask[G];
    g_u64 *man = (g_u64 *)jb.manifest;
    if ((mask >> lane) & 1) {
        const uint64_t below = lane ? (mask & ((1ULL << lane) - 1)) : 0;
        const uint64_t slot = offsets[G] + (uint64_t)__popcll(below);
        list[slot] = ((uint64_t)b << 40) | i;
        man[i] = payload_arena_off + slot * kChunk;
    } else {
        man[i] = jb.parent_manifest ? ((const g_u64 *)jb.parent_manifest)[i]
                                    : jb.parent_slot0 + i * kChunk;
    }
}

// Copies listed dirty chunks into consecutive slots (64 slots per
// workgroup, one whole chunk per step), zero-padding partial chunks.
__global__ __launch_bounds__(256) void k_pack_dirty(const JobBuf *__restrict__ bufs,
                                                    const Run *__restrict__ runs,
                                                    const uint64_t *__restrict__ list,
                                                    const uint64_t *__restrict__ total_ptr,
                                                    uint64_t payload)
{
    const uint64_t total = *total_ptr;
    const uint64_t s0 = (uint64_t)blockIdx.x * kGroupChunks;
    if (s0 >= total) return;
    const uint32_t ns = (uint32_t)umin(kGroupChunks, total - s0);
    const uint32_t x = threadIdx.x * 16;
    for (uint32_t k = 0; k < ns; ++k) {
        const uint64_t e = list[s0 + k];
        const JobBuf &jb = bufs[e >> 40];
        const uint64_t cb = (e & ((1ULL << 40) - 1)) * kChunk;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (cb + x < jb.nbytes) {
            Cursor cur = cursor_seek(runs, jb.run_begin, jb.run_count, jb.nbytes, cb + x);
            if (cb + x + 16 <= jb.nbytes) v = load16(cursor_addr(cur, cb + x));
            else v = load_partial(cursor_addr(cur, cb + x), (uint32_t)(jb.nbytes - cb - x));
        }
        store16(payload + (s0 + k) * kChunk + x, v);
    }
}

// ---------------------------------------------------------------- classify

// One wavefront per bitmap word (= one 64-chunk group of one buffer): chunk
// i differs iff its K replay fingerprints are not all equal; the wave's
// ballot is the word.
__global__ __launch_bounds__(64) void k_classify(const JobBuf *__restrict__ bufs,
                                                 const uint32_t *__restrict__ map,
                                                 const uint64_t *__restrict__ hashes, uint32_t K,
                                                 uint64_t total, uint64_t *__restrict__ bitmap)
{
    const uint64_t G = blockIdx.x;
    const JobBuf &jb = bufs[map[G]];
    const uint32_t lane = threadIdx.x;
    const uint64_t i = (G - jb.group_begin) * kGroupChunks + lane;
    bool differs = false;
    if (i < jb.nchunks) {
        const uint64_t idx = jb.chunk_begin + i;
        const uint64_t h0 = hashes[idx];
        for (uint32_t k = 1; k < K; ++k) differs |= hashes[(uint64_t)k * total + idx] != h0;
    }
    const uint64_t word = __ballot(differs);
    if (lane == 0) bitmap[G] = word;
}

__global__ void k_labels(const JobBuf *__restrict__ bufs, uint32_t nbuf,
                         const uint64_t *__restrict__ bitmap, uint8_t *__restrict__ labels)
{
    const uint32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nbuf) return;
    const JobBuf &jb = bufs[b];
    const uint64_t nw = (jb.nchunks + kGroupChunks - 1) / kGroupChunks;
    uint64_t any = 0;
    for (uint64_t w = 0; w < nw; ++w) any |= bitmap[jb.group_begin + w];
    labels[b] = any ? 1 : 0;
}

}  // namespace

// ---------------------------------------------------------------- launchers

hipError_t launch_group_map(const JobBuf *bufs, uint32_t nbuf, uint64_t ngroups, uint32_t *map,
                            hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((ngroups + 255) / 256);
    hipLaunchKernelGGL(k_group_map, dim3(blocks), dim3(256), 0, s, bufs, nbuf, ngroups, map);
    return hipGetLastError();
}

hipError_t launch_hash(const JobBuf *bufs, const Run *runs, const uint32_t *map, uint64_t ngroups,
                       bool copy, bool diff, uint64_t *nodes, uint32_t *dirty_count,
                       uint64_t *dirty_mask, hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    const dim3 grid((uint32_t)ngroups), block(128);
    if (copy && diff) return hipErrorInvalidValue;
    if (copy)
        hipLaunchKernelGGL((k_hash<true, false>), grid, block, 0, s, bufs, runs, map, nodes, dirty_count, dirty_mask);
    else if (diff)
        hipLaunchKernelGGL((k_hash<false, true>), grid, block, 0, s, bufs, runs, map, nodes, dirty_count, dirty_mask);
    else
        hipLaunchKernelGGL((k_hash<false, false>), grid, block, 0, s, bufs, runs, map, nodes, dirty_count, dirty_mask);
    return hipGetLastError();
}

hipError_t launch_merkle(const MerkleList *lists, uint32_t nlists, const uint64_t *in,
                         uint64_t *scratch_a, uint64_t *scratch_b, uint64_t *roots_out,
                         hipStream_t s)
{
    if (nlists == 0) return hipSuccess;
    hipLaunchKernelGGL(k_merkle, dim3(nlists), dim3(256), 0, s, lists, in, scratch_a, scratch_b, roots_out);
    return hipGetLastError();
}

hipError_t launch_pack(const JobBuf *bufs, const Run *runs, const uint32_t *map, uint64_t ngroups,
                       hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack, dim3((uint32_t)ngroups), dim3(256), 0, s, bufs, runs, map);
    return hipGetLastError();
}

hipError_t launch_restore(const JobBuf *bufs, const Run *runs, const uint32_t *map,
                          uint64_t ngroups, uint64_t arena_base, hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    hipLaunchKernelGGL(k_restore, dim3((uint32_t)ngroups), dim3(256), 0, s, bufs, runs, map, arena_base);
    return hipGetLastError();
}

hipError_t launch_scan(const uint32_t *counts, uint64_t n, uint64_t *offsets, uint64_t *total,
                       hipStream_t s)
{
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, counts, n, offsets, total);
    return hipGetLastError();
}

hipError_t launch_compact(const JobBuf *bufs, const uint32_t *map, uint64_t ngroups,
                          const uint64_t *dirty_mask, const uint64_t *offsets,
                          uint64_t payload_arena_off, uint64_t *list, hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    hipLaunchKernelGGL(k_compact, dim3((uint32_t)ngroups), dim3(64), 0, s, bufs, map, dirty_mask, offsets,
                       payload_arena_off, list);
    return hipGetLastError();
}

hipError_t launch_pack_dirty(const JobBuf *bufs, const Run *runs, const uint64_t *list,
                             const uint64_t *total, uint64_t max_slots, uint64_t payload,
                             hipStream_t s)
{
    if (max_slots == 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((max_slots + kGroupChunks - 1) / kGroupChunks);
    hipLaunchKernelGGL(k_pack_dirty, dim3(blocks), dim3(256), 0, s, bufs, runs, list, total, payload);
    return hipGetLastError();
}

hipError_t launch_classify(const JobBuf *bufs, const uint32_t *map, uint64_t ngroups,
                           const uint64_t *hashes, uint32_t K, uint64_t total, uint64_t *bitmap,
                           hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    hipLaunchKernelGGL(k_classify, dim3((uint32_t)ngroups), dim3(64), 0, s, bufs, map, hashes, K, total, bitmap);
    return hipGetLastError();
}

hipError_t launch_labels(const JobBuf *bufs, uint32_t nbuf, const uint64_t *bitmap,
                         uint8_t *labels, hipStream_t s)
{
    if (nbuf == 0) return hipSuccess;
    hipLaunchKernelGGL(k_labels, dim3((nbuf + 255) / 256), dim3(256), 0, s, bufs, nbuf, bitmap, labels);
    return hipGetLastError();
}

}  // namespace pcs

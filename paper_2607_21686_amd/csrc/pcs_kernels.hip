// pcs_kernels.hip -- gfx950 (CDNA4) kernels of libpcs: chunked XXH64 with a
// Merkle combine, fused pack + fingerprint, scatter restore, incremental
// dirty-chunk packing and cross-replay classification.
//
// Work decomposition shared by every kernel: a job is a table of buffers,
// each cut into 4096-byte chunks, and the chunks of one buffer into aligned
// groups of 64.  One workgroup handles one group (in a job of at most 128
// groups, an eighth of one); it finds its buffer through a group-to-buffer
// map (k_group_map) when the tables live in device memory,
// or by a short search when a small job carries its tables in the kernel
// arguments (no upload and no map launch).  Groups never straddle
// buffers, so a group's 64 chunk fingerprints reduce to one Merkle node
// inside the workgroup (a promote-odd tree over n leaves splits into aligned
// 64-leaf subtrees), and a group is exactly one word of the classification
// bitmap.
//
// Memory traffic is 16-byte vector loads and stores throughout.  Nothing
// here is a contraction, so no MFMA is used; the hash is 64-bit integer
// multiply work on the vector ALU.
#include <hip/hip_ext.h>

#include <algorithm>
#include <type_traits>

#include "pcs_device.h"

// Device scratch of the allocation-free entry point (pcs_fingerprint_noalloc):
// descriptor tables, the group map and the Merkle levels of one call.  Every
// GPU the library runs on holds its own copy until the process ends.  In host
// code this name is a host-side stand-in, never a device address: host code
// uses only the per-device address that static_scratch_address returns.
static __device__ __align__(256) uint8_t scratch[pcs::kStaticScratchBytes];

namespace pcs {

hipError_t static_scratch_address(uint64_t *addr)
{
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    *addr = e == hipSuccess ? (uint64_t)p : 0;
    return e;
}

namespace {

// Timing events for the next kernel launch, set by the runtime around one
// launcher call while dispatch timing is on: that launch stamps `start` when
// its kernel begins and `stop` when it ends (the dispatch's own timestamps,
// so queueing and launch overhead are not counted).  Other launches take the
// plain launch path.
thread_local hipEvent_t t_start = nullptr, t_stop = nullptr;
thread_local bool t_used = false;

template <class K, class... Args>
void run_kernel(K kernel, dim3 grid, dim3 block, hipStream_t s, Args... args)
{
    if (!t_start) {
        hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
        return;
    }
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, t_start, t_stop, 0, args...);
    t_start = t_stop = nullptr;
    t_used = true;
}

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

// The run of [begin, begin + count) that holds logical offset L: the largest
// index whose lstart <= L (runs are sorted by lstart, the first at 0).
__device__ __forceinline__ uint32_t find_run(const Run *runs, uint32_t begin, uint32_t count, uint64_t L)
{
    uint32_t lo = begin, hi = begin + count;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (runs[mid].lstart <= L) lo = mid; else hi = mid;
    }
    return lo;
}

// The tile a workgroup takes (xcd_tile_of).  Measured on MI355X against the
// plain blockIdx order: pack + fingerprint of a 512 MiB ring window 204 ->
// 190-198 us, restore 189 -> 180-185 us; on the 1024-session batch the fused
// kernel 11.5 -> 10.9-11.0 ms in every input placement tried, where
// contiguous eighths alone gave 11.45 ms in some.
__device__ __forceinline__ uint32_t xcd_tile() { return xcd_tile_of(blockIdx.x, gridDim.x); }

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

// Streaming (nontemporal) forms for bulk state that is touched once per call.
__device__ __forceinline__ uint4 load16_nt(uint64_t a)
{
    const v4u32 v = __builtin_nontemporal_load((const g_v4u32 *)a);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store16_nt(uint64_t a, uint4 v)
{
    const v4u32 w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, (g_v4u32 *)a);
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

// One lane per group: its buffer (the largest b with group_begin <= g; empty
// buffers own no group and lose ties) and the run holding its first byte, so
// that the tile kernels start without searching.
__global__ void k_group_map(const JobBuf *__restrict__ bufs, const Run *__restrict__ runs, uint32_t nbuf,
                            uint64_t ngroups, GroupRef *__restrict__ map)
{
    const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= ngroups) return;
    uint32_t lo = 0, hi = nbuf;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (bufs[mid].group_begin <= g) lo = mid; else hi = mid;
    }
    const JobBuf &jb = bufs[lo];
    const uint64_t x0 = (g - jb.group_begin) * kGroupChunks * kChunk;
    map[g] = GroupRef{lo, find_run(runs, jb.run_begin, jb.run_count, x0)};
}

// ---------------------------------------------------------------- fingerprint

// Physical address of logical offset L of a buffer (binary search of its
// runs): the path for the few chunks that straddle a ring wrap.
__device__ uint64_t phys_addr(const Run *runs, uint32_t begin, uint32_t count, uint64_t L)
{
    const Run r = runs[find_run(runs, begin, count, L)];
    return r.addr + (L - r.lstart);
}

// Where one chunk's bytes lie: byte x (x < len) is at (x < split ? a1 : a2)
// + x when the chunk spans at most two physical runs (it straddles a ring's
// wrap, or the end of one ring row set and the start of the next, when that
// boundary falls inside it); a1 = 0 marks a chunk spanning more runs (rows
// shorter than a chunk), whose addresses are searched per access.  Run
// boundaries are 16-byte aligned, so no 16-byte granule crosses one.
struct ChunkLoc {
    uint64_t a1, a2;
    uint32_t split, len;
};

// Per-chunk setup shared by the tile kernels: lane c < 64 of the first
// wavefront describes chunk c of the group.  r0 is the run holding the
// group's first byte; a chunk's run is found by stepping forward from there
// (a group usually lies in one or two runs), with a search for groups that
// span many short runs.
__device__ __forceinline__ void chunk_table(const JobBuf &jb, const Run *runs, uint32_t r0, uint64_t c0,
                                            uint32_t nv, ChunkLoc *loc)
{
    const uint32_t t = threadIdx.x;
    if (t < kGroupChunks) {
        ChunkLoc l{0, 0, 0, 0};
        if (t < nv) {
            const uint64_t cb = (c0 + t) * kChunk;
            l.len = (uint32_t)umin(kChunk, jb.nbytes - cb);
            const uint32_t last = jb.run_begin + jb.run_count - 1;
            uint32_t idx = r0;
            Run r = runs[idx];
            uint64_t end = idx < last ? runs[idx + 1].lstart : jb.nbytes;
            for (int k = 0; end <= cb; ++k) {  // cb < nbytes: ends at the last run at the latest
                if (k == 2) {
                    idx = find_run(runs, idx + 1, last - idx, cb);
                } else {
                    ++idx;
                }
                r = runs[idx];
                end = idx < last ? runs[idx + 1].lstart : jb.nbytes;
            }
            const uint64_t a1 = r.addr + (cb - r.lstart);
            if (cb + l.len <= end) {
                l.a1 = l.a2 = a1;
                l.split = l.len;
            } else {  // idx < last here, since the last run ends at nbytes
                const Run r2 = runs[idx + 1];
                const uint64_t end2 = idx + 1 < last ? runs[idx + 2].lstart : jb.nbytes;
                if (cb + l.len <= end2) {
                    l.a1 = a1;
                    l.split = (uint32_t)(end - cb);
                    l.a2 = r2.addr - l.split;  // byte `split` of the chunk is r2's first byte
                }
            }
        }
        loc[t] = l;
    }
}

// Selects word i (0..3) of a 32-byte tail held in registers.
__device__ __forceinline__ uint64_t sel4(uint64_t a, uint64_t b, uint64_t c, uint64_t d, uint32_t i)
{
    return i == 0 ? a : i == 1 ? b : i == 2 ? c : d;
}

// A workgroup's buffer: through the map, or by searching a table of at most
// kArgBufs buffers (largest b with group_begin <= G; empty buffers lose ties).
__device__ __forceinline__ uint32_t buf_index(const DevTables &t, uint64_t G) { return t.map[G].buf; }
__device__ __forceinline__ uint32_t buf_index(const ArgTables &t, uint64_t G)
{
    uint32_t lo = 0, hi = t.nbuf;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (t.bufs[mid].group_begin <= G) lo = mid; else hi = mid;
    }
    return lo;
}

// A workgroup's buffer and the run holding its group's first byte.
__device__ __forceinline__ GroupRef group_ref(const DevTables &t, uint64_t G) { return t.map[G]; }
__device__ __forceinline__ GroupRef group_ref(const ArgTables &t, uint64_t G)
{
    const uint32_t b = buf_index(t, G);
    const JobBuf &jb = t.bufs[b];
    return GroupRef{b, find_run(t.runs, jb.run_begin, jb.run_count, (G - jb.group_begin) * kGroupChunks * kChunk)};
}

// First-round stagger.  The workgroups of a launch's first round (one per CU)
// all start together and then move their slices in step: every CU reads the
// same offsets within its chunks at the same moment.  In jobs of a few
// rounds this costs the first two rounds about a fifth of their speed
// (per-workgroup timelines on MI355X, 512 MiB pack + fingerprint: 25 against
// 21 us per group; jobs of 768 MiB and more do not show it).  Holding the
// first-round workgroups back by 0..7 phases of stg.ticks of the constant
// real-time counter (phase = position within the XCD, mod 8) spreads them
// over most of a group's duration; later workgroups start whenever a CU
// frees up and need no stagger.  The wait is also bounded by a spin count,
// so it ends even if the counter stood still.
__device__ __forceinline__ void stagger_start(const Stagger &stg)
{
    if (stg.ticks == 0 || blockIdx.x >= stg.first_round) return;
    const uint64_t wait = (uint64_t)((blockIdx.x / kXcds) % kStaggerPhases) * stg.ticks;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (uint32_t spin = 0; spin < kStaggerMaxSpins && __builtin_amdgcn_s_memrealtime() - t0 < wait; ++spin)
        __builtin_amdgcn_s_sleep(2);
}

// Fingerprint tile kernels (k_hash, k_hash_staggered; the body is
// hash_tile).  One workgroup = one tile of CPW chunks of one
// buffer: a whole 64-chunk group, or for small jobs an eighth of one, so
// that a few groups still occupy many CUs (the tile's Merkle node is then an
// aligned 8-chunk subtree).  Step k moves the k-th SL-byte slice of every
// chunk of the tile:
// all T lanes load it with coalesced 16-byte loads (SL/16 lanes per chunk
// slice), kModePack stores it to the chunk's snapshot slot (zero-padding a
// partial last chunk) and kModeVerify to the buffer's runs, and every lane
// writes it to an LDS tile; then lane quads of the first 4*CPW lanes hash
// the tile while the next slice's loads are in flight.  Lane q of a quad owns
// XXH64 accumulator q, which reads exactly bytes [8q, 8q+8) of each 32-byte
// stripe.  A wavefront issues a lane's rounds one after another (a round is
// about ten instructions, most of them 32-bit multiply steps of the 64-bit
// products), so one accumulator per lane halves the instructions a chunk's
// chain costs each wavefront and spreads the hashing over twice as many
// wavefronts as lane pairs with two accumulators each would.  kModeDiff /
// kModeVerify ballot one flag per chunk into a per-group mask (the group is
// one bitmap word; a diff sub-tile writes its byte of the word).  WB: the
// pack stores go through the caches (write-back) instead of streaming past
// them; see kPackWriteBackMaxRounds.
template <class Tab, int MODE, int T, int SL, int CPW, bool STAGGER, bool WB>
__device__ __forceinline__ void hash_tile(const Tab &tab, uint64_t *__restrict__ nodes,
                                          uint64_t *__restrict__ flag_mask, uint64_t arena_base, const Stagger &stg)
{
    constexpr uint32_t kSteps = kChunk / SL;
    constexpr uint32_t kRow = SL + 32;                  // padded LDS row: the quads of 8 chunks hit distinct banks
    constexpr uint32_t LPS = SL / 16;                   // lanes per chunk slice
    constexpr int U = CPW * SL / 16 / T;                // granules per lane per step
    constexpr uint32_t kTiles = kGroupChunks / CPW;     // tiles per 64-chunk group
    constexpr bool kFromSlots = MODE == kModeVerify;    // source is the snapshot, destination the runs
    static_assert(U >= 1 && T % LPS == 0 && kGroupChunks % CPW == 0, "tile shape");
    static_assert(T >= 4 * CPW, "one lane per accumulator");
    static_assert(CPW == kGroupChunks || MODE != kModeVerify, "verify flags need whole groups");
    static_assert(CPW == kGroupChunks || CPW == 8 || MODE != kModeDiff, "a diff sub-tile writes one mask byte");
    __shared__ __attribute__((aligned(16))) uint8_t tile[CPW * kRow];
    __shared__ ChunkLoc cloc[kGroupChunks];
    __shared__ uint64_t leaves[CPW];
    __shared__ uint32_t dflag[CPW];

    const uint32_t tile_id = xcd_tile();
    if constexpr (STAGGER) stagger_start(stg);
    const uint64_t G = tile_id / kTiles;
    const GroupRef gr = group_ref(tab, G);
    const JobBuf &jb = tab.bufs[gr.buf];
    const Run *runs = tab.runs;
    const uint32_t t = threadIdx.x;
    const uint64_t c0 = (G - jb.group_begin) * kGroupChunks + (tile_id % kTiles) * CPW;
    if (c0 >= jb.nchunks) {  // a buffer's last group may end before this tile
        // A diff sub-tile owns byte (tile % 8) of its group's dirty mask:
        // an empty one writes it as 0 so every byte of the mask is defined.
        if (MODE == kModeDiff && kTiles > 1 && t == 0 && flag_mask)
            ((g_u8 *)flag_mask)[G * kTiles + tile_id % kTiles] = 0;
        return;
    }
    const uint32_t nv = (uint32_t)umin(CPW, jb.nchunks - c0);
    const uint32_t run_begin = jb.run_begin, run_count = jb.run_count;
    const g_u64 *man = (const g_u64 *)jb.manifest;
    chunk_table(jb, runs, gr.run, c0, nv, cloc);
    __syncthreads();

    // This lane's granules: chunk (k*T + t) / LPS, slot t % LPS of each slice.
    const uint32_t slot = (t % LPS) * 16;
    uint64_t ga[U], gb[U];  // runs side: where the chunk's bytes lie (ChunkLoc)
    uint64_t sa[U];         // slots side: the chunk's 4096-byte slot (0 if the group has no such chunk)
    uint32_t gs[U], gl[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const uint32_t c = (k * T + t) / LPS;
        const ChunkLoc l = c < nv ? cloc[c] : ChunkLoc{0, 0, 0, 0};
        ga[k] = l.a1;
        gb[k] = l.a2;
        gs[k] = l.split;
        gl[k] = l.len;
        sa[k] = 0;
        if (c < nv && (MODE == kModePack || kFromSlots))
            sa[k] = (kFromSlots && man) ? arena_base + man[c0 + c] : jb.payload + (c0 + c) * kChunk;
    }
    auto runs_addr = [&](int k, uint32_t x) -> uint64_t {
        const uint32_t c = (k * T + t) / LPS;
        return ga[k] ? (x < gs[k] ? ga[k] : gb[k]) + x : phys_addr(runs, run_begin, run_count, (c0 + c) * kChunk + x);
    };
    auto load_granule = [&](int k, uint32_t x) -> uint4 {
        uint4 v = make_uint4(0, 0, 0, 0);
        if (x < gl[k]) {
            if (kFromSlots) {
                v = load16_nt(sa[k] + x);  // slots are whole 4096-byte granules, zero padded
            } else {
                const uint64_t a = runs_addr(k, x);
                v = x + 16 <= gl[k] ? load16_nt(a) : load_partial(a, gl[k] - x);
            }
        }
        return v;
    };

    uint4 r[U];
#pragma unroll
    for (int k = 0; k < U; ++k) r[k] = load_granule(k, slot);

    const uint32_t ci = t >> 2, q = t & 3;
    const bool hasher = t < 4 * CPW && ci < nv;
    const uint32_t len = hasher ? cloc[ci].len : 0;
    const uint32_t nst = len >> 5;
    // Incremental checkpoint: where the parent holds this chunk, fetched now
    // and entered in the new manifest at the end if the chunk is clean (a
    // dirty chunk's entry is its slot, written once the slots are placed).
    uint64_t parent_loc = 0;
    if (MODE == kModeDiff && hasher && q == 0 && jb.manifest && c0 + ci < jb.parent_chunks)
        parent_loc = jb.parent_manifest ? ((const g_u64 *)jb.parent_manifest)[c0 + ci]
                                        : jb.parent_slot0 + (c0 + ci) * kChunk;
    // Accumulator q with seed 0: P1 + P2, P2, 0, -P1.
    uint64_t va = q == 0 ? P1 + P2 : q == 1 ? P2 : q == 2 ? 0 : 0 - P1;
    uint64_t tw0 = 0, tw1 = 0, tw2 = 0, tw3 = 0;  // the chunk's tail (< 32 bytes), zero padded

    for (uint32_t step = 0; step < kSteps; ++step) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const uint32_t c = (k * T + t) / LPS;
            if (c < nv) {
                const uint32_t x = step * SL + slot;
                if (MODE == kModePack) {
                    if (WB) store16(sa[k] + x, r[k]);
                    else store16_nt(sa[k] + x, r[k]);
                }
                if (kFromSlots && x < gl[k]) {
                    if (x + 16 <= gl[k]) store16_nt(runs_addr(k, x), r[k]);
                    else store_partial(runs_addr(k, x), r[k], gl[k] - x);
                }
                *reinterpret_cast<uint4 *>(tile + c * kRow + slot) = r[k];
            }
        }
        __syncthreads();
        if (step + 1 < kSteps) {
#pragma unroll
            for (int k = 0; k < U; ++k) r[k] = load_granule(k, (step + 1) * SL + slot);
        }
        if (hasher) {
            const uint8_t *row = tile + ci * kRow;
            const uint32_t s0 = step * (SL / 32);
            const uint32_t ns = nst > s0 ? umin(SL / 32, nst - s0) : 0;
#pragma unroll 8
            for (uint32_t s = 0; s < ns; ++s) {
                const uint2 d = *reinterpret_cast<const uint2 *>(row + 32 * s + 8 * q);
                va = xround(va, ((uint64_t)d.y << 32) | d.x);
            }
            const uint32_t tp = nst * 32;  // tail start, 32-aligned, inside this slice if here
            if (q == 0 && tp < len && tp >= step * SL && tp < (step + 1) * SL) {
                const uint4 x = *reinterpret_cast<const uint4 *>(row + tp - step * SL);
                const uint4 y = *reinterpret_cast<const uint4 *>(row + tp - step * SL + 16);
                tw0 = ((uint64_t)x.y << 32) | x.x;
                tw1 = ((uint64_t)x.w << 32) | x.z;
                tw2 = ((uint64_t)y.y << 32) | y.x;
                tw3 = ((uint64_t)y.w << 32) | y.z;
            }
        }
        __syncthreads();
    }

    if (t < 4 * CPW) {
        // Accumulators 1-3 of a quad to its lane 0 (a quad never straddles
        // a wavefront).
        const uint64_t v2 = shfl64(va, (int)(t + 1) & 63);
        const uint64_t v3 = shfl64(va, (int)(t + 2) & 63);
        const uint64_t v4 = shfl64(va, (int)(t + 3) & 63);
        if (hasher && q == 0) {
            uint64_t acc;
            if (len >= 32) {
                acc = rotl(va, 1) + rotl(v2, 7) + rotl(v3, 12) + rotl(v4, 18);
                acc = xmerge(acc, va);
                acc = xmerge(acc, v2);
                acc = xmerge(acc, v3);
                acc = xmerge(acc, v4);
            } else {
                acc = P5;
            }
            acc += len;
            // Tail: 8-byte lanes, one 4-byte lane, single bytes (offsets
            // relative to the tail start).
            uint32_t o = 0;
            const uint32_t rem = len - nst * 32;
            for (; rem - o >= 8; o += 8) {
                acc ^= xround(0, sel4(tw0, tw1, tw2, tw3, o >> 3));
                acc = rotl(acc, 27) * P1 + P4;
            }
            if (rem - o >= 4) {
                acc ^= (uint64_t)(uint32_t)sel4(tw0, tw1, tw2, tw3, o >> 3) * P1;
                acc = rotl(acc, 23) * P2 + P3;
                o += 4;
            }
            for (; o < rem; ++o) {
                const uint64_t byte = (sel4(tw0, tw1, tw2, tw3, o >> 3) >> (8 * (o & 7))) & 0xFF;
                acc ^= byte * P5;
                acc = rotl(acc, 11) * P1;
            }
            const uint64_t h = avalanche(acc);
            const uint64_t i = c0 + ci;
            if (jb.hash_dst[0]) ((g_u64 *)jb.hash_dst[0])[i] = h;
            if (jb.hash_dst[1]) ((g_u64 *)jb.hash_dst[1])[i] = h;
            leaves[ci] = h;
            if (MODE == kModeDiff) {
                const bool d = i >= jb.parent_chunks || ((const g_u64 *)jb.parent_hash)[i] != h;
                dflag[ci] = d ? 1u : 0u;
                if (!d && jb.manifest) ((g_u64 *)jb.manifest)[i] = parent_loc;
            }
            if (MODE == kModeVerify) dflag[ci] = ((const g_u64 *)jb.parent_hash)[i] != h ? 1u : 0u;
        }
    }
    __syncthreads();
    if (t < 64) {
        const uint64_t v = t < nv ? leaves[t] : 0;
        const uint64_t root = wave_merkle(v, nv);
        if (t == 0 && nodes) nodes[tile_id] = root;  // the tile's Merkle node (an aligned subtree)
        if (MODE == kModeDiff || MODE == kModeVerify) {
            // Bit c of group G's mask = chunk c of the group; a sub-tile
            // writes its 8 bits as byte (tile % 8) of the little-endian word.
            const uint64_t mask = __ballot(t < nv && dflag[t] != 0);
            if (t == 0 && flag_mask) {
                if (kTiles == 1) flag_mask[G] = mask;
                else ((g_u8 *)flag_mask)[G * kTiles + tile_id % kTiles] = (uint8_t)mask;
            }
        }
    }
}

template <class Tab, int MODE, int T, int SL, int CPW, bool WB>
__global__ __launch_bounds__(T) void k_hash(const Tab tab, uint64_t *__restrict__ nodes,
                                            uint64_t *__restrict__ flag_mask, uint64_t arena_base)
{
    hash_tile<Tab, MODE, T, SL, CPW, false, WB>(tab, nodes, flag_mask, arena_base, Stagger{0, 0});
}

// k_hash with the first-round stagger (pack and verify jobs of a few rounds):
// a kernel of its own, so the others keep their code and arguments.  Its
// jobs are all within the write-back bound, so a pack stores write-back.
template <class Tab, int MODE, int T, int SL, int CPW>
__global__ __launch_bounds__(T) void k_hash_staggered(const Tab tab, uint64_t *__restrict__ nodes,
                                                      uint64_t *__restrict__ flag_mask, uint64_t arena_base,
                                                      Stagger stg)
{
    hash_tile<Tab, MODE, T, SL, CPW, true, MODE == kModePack>(tab, nodes, flag_mask, arena_base, stg);
}

// ---------------------------------------------------------------- Merkle lists

// Promote-odd Merkle root of src[0, m), computed by the whole workgroup
// (NT lanes; pre: the first level of a list of more than 4096 values is
// already in sa); the result is valid in thread 0.  Aligned 64-value blocks
// reduce independently (one wavefront each); up to two passes through global
// scratch sa/sb (each read only after it is fully written) bring the list to
// <= 4096 values, then the rest happens in LDS.  Ends with a barrier so the
// LDS buffers can be reused.
template <int NT>
__device__ uint64_t reduce_list(const uint64_t *src, uint64_t m, uint64_t *sa, uint64_t *sb, uint64_t *lds,
                                uint64_t *lds2, bool pre)
{
    constexpr uint32_t NW = NT / 64;  // wavefronts
    const uint32_t t = threadIdx.x, wave = t >> 6, lane = t & 63;
    uint64_t root = 0;
    if (m == 0) {
        root = empty_hash();
    } else {
        uint64_t *scratch[2] = {sa, sb};
        for (int k = 0; k < 2 && m > 4096; ++k) {
            // Four blocks per wavefront in flight: their loads issue before
            // the first reduction (a scheduling barrier keeps them there).
            // pre: the first level is already in sa (k_merkle_blocks).
            const uint64_t nb = (m + 63) / 64;
            for (uint64_t blk0 = wave; blk0 < nb && !(pre && k == 0); blk0 += 4 * NW) {
                uint64_t v[4];
                uint32_t cnt[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const uint64_t blk = blk0 + u * NW;
                    cnt[u] = blk < nb ? (uint32_t)umin(64, m - 64 * blk) : 0;
                    v[u] = lane < cnt[u] ? src[64 * blk + lane] : 0;
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (!cnt[u]) continue;
                    const uint64_t r = wave_merkle(v[u], cnt[u]);
                    if (lane == 0) scratch[k][blk0 + u * NW] = r;
                }
            }
            __syncthreads();
            src = scratch[k];
            m = nb;
        }
        for (uint64_t j = t; j < m; j += NT) lds[j] = src[j];
        __syncthreads();
        const uint64_t *ls = lds;
        if (m > 64) {
            const uint64_t nb = (m + 63) / 64;
            for (uint64_t blk = wave; blk < nb; blk += NW) {
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
    __syncthreads();
    return root;
}

// One workgroup per list (device-memory list table); NT lanes (1024 when a
// list is long enough to need passes through memory, else 256).
template <int NT>
__global__ __launch_bounds__(NT) void k_merkle(const MerkleList *__restrict__ lists,
                                               const uint64_t *__restrict__ in,
                                               uint64_t *__restrict__ sa, uint64_t *__restrict__ sb,
                                               uint64_t *__restrict__ roots_out, bool pre)
{
    __shared__ uint64_t lds[4096];
    __shared__ uint64_t lds2[64];
    const MerkleList Lst = lists[blockIdx.x];
    const uint64_t root =
        reduce_list<NT>(in + Lst.begin, Lst.count, sa + Lst.begin, sb + Lst.begin, lds, lds2, pre);
    if (threadIdx.x == 0) {
        if (Lst.dst[0]) *(g_u64 *)Lst.dst[0] = root;
        if (Lst.dst[1]) *(g_u64 *)Lst.dst[1] = root;
        if (roots_out) roots_out[blockIdx.x] = root;
    }
}

// Promote-odd Merkle root of ls[0, m) already in LDS (m <= 4096), computed
// by the workgroup (NT lanes); valid in thread 0.  Ends with a barrier.
template <int NT>
__device__ uint64_t reduce_lds(const uint64_t *ls, uint64_t m, uint64_t *lds2)
{
    constexpr uint32_t NW = NT / 64;
    const uint32_t t = threadIdx.x, wave = t >> 6, lane = t & 63;
    uint64_t root = 0;
    if (m == 0) {
        root = empty_hash();
    } else {
        if (m > 64) {
            const uint64_t nb = (m + 63) / 64;
            for (uint64_t blk = wave; blk < nb; blk += NW) {
                const uint32_t cnt = (uint32_t)umin(64, m - 64 * blk);
                const uint64_t v = lane < cnt ? ls[64 * blk + lane] : 0;
                const uint64_t r = wave_merkle(v, cnt);
                if (lane == 0) lds2[blk] = r;
            }
            __syncthreads();
            ls = lds2;
            m = nb;
        }
        if (wave == 0) root = wave_merkle(lane < m ? ls[lane] : 0, (uint32_t)m);
    }
    __syncthreads();
    return root;
}

// The lists of a small job, reduced by one workgroup of NT lanes: every
// buffer list, then every session list over the buffer roots just computed
// (kept in LDS).  Buffer lists that follow each other in `in` and hold at
// most 4096 values together (a job's buffers, the usual case) are loaded
// into LDS in one pass, so the lists wait on one round trip to memory, not
// one each.  Ends with a barrier.
template <int NT>
__device__ void merkle_lists(const ArgLists &L, const uint64_t *in, uint64_t *sa, uint64_t *sb, uint64_t *lds,
                             uint64_t *lds2, uint64_t *roots, bool pre = false)
{
    bool one_pass = L.nbuf_lists > 0;
    const uint64_t lo = one_pass ? L.lists[0].begin : 0;
    uint64_t hi = lo;
    for (uint32_t j = 0; j < L.nbuf_lists; ++j) {
        one_pass = one_pass && L.lists[j].begin == hi;
        hi = L.lists[j].begin + L.lists[j].count;
    }
    one_pass = one_pass && hi - lo <= 4096;
    if (one_pass) {
        for (uint64_t j = threadIdx.x; j < hi - lo; j += NT) lds[j] = in[lo + j];
        __syncthreads();
    }
    for (uint32_t j = 0; j < L.nbuf_lists; ++j) {
        const MerkleList &Lst = L.lists[j];
        const uint64_t root =
            one_pass ? reduce_lds<NT>(lds + (Lst.begin - lo), Lst.count, lds2)
                     : reduce_list<NT>(in + Lst.begin, Lst.count, sa + Lst.begin, sb + Lst.begin, lds, lds2, pre);
        if (threadIdx.x == 0) {
            roots[j] = root;
            if (Lst.dst[0]) *(g_u64 *)Lst.dst[0] = root;
            if (Lst.dst[1]) *(g_u64 *)Lst.dst[1] = root;
        }
    }
    __syncthreads();
    if (threadIdx.x < 64) {
        const uint32_t lane = threadIdx.x;
        for (uint32_t j = L.nbuf_lists; j < L.nlists; ++j) {
            const MerkleList &Lst = L.lists[j];
            const uint32_t cnt = (uint32_t)Lst.count;
            const uint64_t v = lane < cnt ? roots[Lst.begin + lane] : 0;
            const uint64_t root = cnt ? wave_merkle(v, cnt) : empty_hash();
            if (lane == 0) {
                if (Lst.dst[0]) *(g_u64 *)Lst.dst[0] = root;
                if (Lst.dst[1]) *(g_u64 *)Lst.dst[1] = root;
            }
        }
    }
    __syncthreads();
}

// One workgroup for a small job's Merkle lists.
__global__ __launch_bounds__(1024) void k_merkle_small(const ArgLists L, const uint64_t *__restrict__ in,
                                                       uint64_t *__restrict__ sa, uint64_t *__restrict__ sb, bool pre)
{
    __shared__ uint64_t lds[4096];
    __shared__ uint64_t lds2[64];
    __shared__ uint64_t roots[kArgBufs];
    merkle_lists<1024>(L, in, sa, sb, lds, lds2, roots, pre);
}

// Grid-wide first level of long Merkle lists (LongLists): wavefront w
// reduces aligned 64-value block w - block_begin[j] of list j into
// sa[begin[j] + block], where the list's own reduction would have put it.
__global__ __launch_bounds__(256) void k_merkle_blocks(const LongLists L, const uint64_t *__restrict__ in,
                                                       uint64_t *__restrict__ sa)
{
    const uint64_t w = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    if (w >= L.block_begin[L.n]) return;
    uint32_t j = 0;
    while (j + 1 < L.n && L.block_begin[j + 1] <= w) ++j;
    const uint64_t blk = w - L.block_begin[j];
    const uint32_t cnt = (uint32_t)umin(64, L.count[j] - 64 * blk);
    const uint64_t v = lane < cnt ? in[L.begin[j] + 64 * blk + lane] : 0;
    const uint64_t r = wave_merkle(v, cnt);
    if (lane == 0) sa[L.begin[j] + blk] = r;
}

// ---------------------------------------------------------------- copies

// Copy tile kernel: one workgroup moves one tile of CPW chunks (a 64-chunk
// group, or an eighth of one in small jobs), SL bytes of every chunk per
// step, with coalesced 16-byte loads and stores: the fused kernel's tile
// without the hash and the LDS staging, in a shape of its own (512 lanes and
// 1 KiB slices for whole groups, measured faster for copies than the fused
// kernel's 1024 lanes and 512-byte slices).
//   PACK:    the buffer's runs -> the chunk slots of the snapshot; a partial
//            last chunk is zero-padded to the end of its slot.
//   !PACK:   the chunk slots (contiguous, or per chunk through a manifest of
//            arena offsets) -> the destination buffer's runs; only logical
//            bytes are written.
template <class Tab, bool PACK, int T, int SL, int CPW>
__global__ __launch_bounds__(T) void k_copy(const Tab tab, uint64_t arena_base, bool wb)
{
    constexpr uint32_t kSteps = kChunk / SL, LPS = SL / 16;
    constexpr int U = CPW * SL / 16 / T;
    constexpr uint32_t kTiles = kGroupChunks / CPW;
    static_assert(U >= 1 && T % LPS == 0 && kGroupChunks % CPW == 0, "tile shape");
    __shared__ ChunkLoc cloc[kGroupChunks];
    const uint32_t tile_id = xcd_tile();
    const uint64_t G = tile_id / kTiles;
    const GroupRef gr = group_ref(tab, G);
    const JobBuf &jb = tab.bufs[gr.buf];
    const Run *runs = tab.runs;
    const uint32_t t = threadIdx.x;
    const uint64_t c0 = (G - jb.group_begin) * kGroupChunks + (tile_id % kTiles) * CPW;
    if (c0 >= jb.nchunks) return;  // a buffer's last group may end before this tile
    const uint32_t nv = (uint32_t)umin(CPW, jb.nchunks - c0);
    const uint32_t run_begin = jb.run_begin, run_count = jb.run_count;
    const g_u64 *man = (const g_u64 *)jb.manifest;
    chunk_table(jb, runs, gr.run, c0, nv, cloc);
    __syncthreads();

    const uint32_t slot = (t % LPS) * 16;
    uint64_t ra[U], rb[U], sa[U];
    uint32_t rs[U], gl[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const uint32_t c = (k * T + t) / LPS;
        const ChunkLoc l = c < nv ? cloc[c] : ChunkLoc{0, 0, 0, 0};
        ra[k] = l.a1;
        rb[k] = l.a2;
        rs[k] = l.split;
        gl[k] = l.len;
        sa[k] = c < nv ? (PACK || !man ? jb.payload + (c0 + c) * kChunk : arena_base + man[c0 + c]) : 0;
    }
    auto runs_addr = [&](int k, uint32_t x) -> uint64_t {
        const uint32_t c = (k * T + t) / LPS;
        return ra[k] ? (x < rs[k] ? ra[k] : rb[k]) + x : phys_addr(runs, run_begin, run_count, (c0 + c) * kChunk + x);
    };
    auto load = [&](int k, uint32_t x) -> uint4 {
        uint4 v = make_uint4(0, 0, 0, 0);
        if (x < gl[k]) {
            if (PACK) v = x + 16 <= gl[k] ? load16_nt(runs_addr(k, x)) : load_partial(runs_addr(k, x), gl[k] - x);
            else v = load16_nt(sa[k] + x);  // slots are whole 4096-byte granules
        }
        return v;
    };
    // The lanes move the tile in lockstep steps (a barrier per step); the
    // next step's loads are issued before this step's stores.  Chunk c moves
    // its slices in an order rotated by c and the tile index, so that a
    // step's accesses cover every offset within a chunk instead of one (all
    // tiles touching the same offsets at once loads the HBM channels
    // unevenly): restores of flat buffers are 3-8% faster with the rotation,
    // the 1024-session batch 1.5% slower.
    uint4 v[U], n[U];
    auto off = [&](int k, uint32_t step) -> uint32_t {
        const uint32_t c = (k * T + t) / LPS;
        return ((step + c + tile_id) % kSteps) * SL + slot;
    };
#pragma unroll
    for (int k = 0; k < U; ++k) v[k] = load(k, off(k, 0));
    for (uint32_t step = 0; step < kSteps; ++step) {
        if (step + 1 < kSteps) {
#pragma unroll
            for (int k = 0; k < U; ++k) n[k] = load(k, off(k, step + 1));
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const uint32_t x = off(k, step);
            if (PACK) {  // wb: write-back stores (jobs within kPackWriteBackMaxRounds)
                if (sa[k]) {
                    if (wb) store16(sa[k] + x, v[k]);
                    else store16_nt(sa[k] + x, v[k]);
                }
            } else if (x < gl[k]) {
                if (x + 16 <= gl[k]) store16_nt(runs_addr(k, x), v[k]);
                else store_partial(runs_addr(k, x), v[k], gl[k] - x);
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < U; ++k) v[k] = n[k];
    }
}

// ---------------------------------------------------------------- incremental

// Inclusive prefix sum across the 64 lanes of a wavefront, in DPP moves (no
// LDS round trips): shifts by 1, 2, 4 and 8 lanes within each row of 16
// lanes, then row 0's total (lane 15) into row 1 and row 2's into row 3
// (row_bcast:15), then rows 0-1's total (lane 31) into rows 2 and 3
// (row_bcast:31).  A lane whose source lies outside its row, or a row the
// row mask leaves out, adds 0 (the `old` operand).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x)
{
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return x;
}

// A scan's entry j: the number of set bits of the 64-bit dirty mask of
// group j of an incremental checkpoint.
struct MaskBits {
    const uint64_t *p;
    __device__ uint64_t operator()(uint64_t j) const { return (uint64_t)__popcll(p[j]); }
};

// Exclusive scan of n counts (one workgroup; Hillis-Steele over 1024
// per-thread partial sums).  Writes offsets[] and *total; returns nothing
// else.  `offsets` may be LDS or global memory.
template <class Count>
__device__ void scan_counts(const Count counts, uint64_t n, uint64_t *offsets, uint64_t *total,
                            uint64_t (*sums)[1024])
{
    const uint32_t t = threadIdx.x;
    const uint64_t per = (n + 1023) / 1024;
    const uint64_t s0 = umin(n, t * per), s1 = umin(n, s0 + per);
    uint64_t s = 0;
    for (uint64_t j = s0; j < s1; ++j) s += counts(j);
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
        run += counts(j);
    }
    if (t == 1023) *total = sums[cur][t];
    __syncthreads();
}

// Thread 1023 of a scan of dirty masks, once the stored-chunk count is
// known: takes this call's payload top from the bump word (bump_now, loaded
// when the kernel started; or sb.reset), writes it lowered by the count's
// slots to the next call's bump word, then publishes the count and the top
// to the host words.  Returns the top (0 when sb.bump is null: the host
// sets the top itself once it has read the count).
__device__ uint64_t place_slots(const SlotBump &sb, uint64_t count, uint64_t bump_now)
{
    uint64_t top = 0;
    if (sb.bump) {
        top = sb.reset ? sb.reset : bump_now;
        *sb.bump_out = top - count * kChunk;
        *sb.top_out = top;
    }
    if (sb.host) {
        ((volatile uint64_t *)sb.host)[0] = count;
        ((volatile uint64_t *)sb.host)[1] = top;
        __threadfence_system();
    }
    return top;
}

// Exclusive scan of counts (offsets and total); for the dirty masks of an
// incremental checkpoint also the placement of its slots (place_slots).
template <class Count>
__global__ __launch_bounds__(1024) void k_scan(const Count counts, uint64_t n, uint64_t *__restrict__ offsets,
                                               uint64_t *__restrict__ total, const SlotBump sb)
{
    __shared__ uint64_t sums[2][1024];
    const uint64_t bump_now = threadIdx.x == 1023 && sb.bump && !sb.reset ? *sb.bump : 0;
    scan_counts(counts, n, offsets, total, sums);
    if (threadIdx.x == 1023) place_slots(sb, *total, bump_now);
}

// Exclusive scan of the dirty masks' set bits of a small incremental job
// (at most kScanCompactMaxGroups groups): thread t holds the masks of groups
// 4t .. 4t+3 (0 past the job), loaded when the kernel started; DPP
// wavefront scans, then one over the 16 wavefront totals (counts stay below
// 2^32).  Writes offsets[] (LDS or global) and returns the total in every
// thread.  Ends with a barrier.
__device__ uint64_t scan_masks_small(const uint64_t (&mk)[4], uint64_t ngroups, uint64_t *offsets, uint32_t *wsum)
{
    const uint32_t t = threadIdx.x, wave = t >> 6, lane = t & 63;
    uint32_t c[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        c[k] = (uint32_t)__popcll(mk[k]);
        sum += c[k];
    }
    const uint32_t incl = wave_incl_scan(sum);
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const uint32_t w = lane < 16 ? wsum[lane] : 0;
        const uint32_t wi = wave_incl_scan(w);
        if (lane < 16) wsum[16 + lane] = wi - w;
        if (lane == 15) wsum[32] = wi;
    }
    __syncthreads();
    uint64_t run = incl - sum + wsum[16 + wave];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (4 * t + k < ngroups) offsets[4 * t + k] = run;
        run += c[k];
    }
    const uint64_t total = wsum[32];
    __syncthreads();
    return total;
}

// Moves chunk i of buffer jb (its logical bytes, zero-padded to 4096) to
// device address dst: the 64 lanes of a wavefront, 64 bytes each, four
// 16-byte loads in flight per lane.
template <class Tab>
__device__ __forceinline__ void copy_chunk(const Tab &tab, const JobBuf &jb, uint64_t i, uint64_t dst, uint32_t lane)
{
    const uint64_t cb = i * kChunk;
    const uint64_t len = umin(kChunk, jb.nbytes - cb);
    uint4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t x = (k * 64 + lane) * 16;
        v[k] = make_uint4(0, 0, 0, 0);
        if (x < len) {
            const uint64_t a = phys_addr(tab.runs, jb.run_begin, jb.run_count, cb + x);
            v[k] = x + 16 <= len ? load16(a) : load_partial(a, (uint32_t)(len - x));
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) store16(dst + (k * 64 + lane) * 16, v[k]);
}

// Small incremental jobs (tables in the kernel arguments, at most
// kScanCompactMaxGroups groups), after the fingerprint + diff tiles, in one
// launch of 1024-lane workgroups that need nothing from one another.
// Workgroup 0 reduces the Merkle lists (buffer and session roots), scans
// the dirty masks' set bits and publishes the stored-chunk count and the
// payload top (place_slots: *total, the next call's bump word, the host
// words).  Every other workgroup scans the masks itself (at most 4096
// words, the same for all, so mostly from L2) into LDS and takes the top
// from *bump.bump, which only an earlier launch wrote; its wavefront w
// then stores slots w, w + stride, ...: slot s belongs to the last group
// whose exclusive offset is at most s (a group with no dirty chunk shares
// its offset with the next group, so the last such group holds s), and
// within it to the dirty chunk with s - offset dirty chunks below it.
// Slots therefore follow (buffer, chunk) order, as k_place_dirty assigns
// them.  Lane 0 enters the slot in the manifest (clean chunks' entries
// were written by the diff tiles) and the wavefront copies the chunk.
__global__ __launch_bounds__(1024) void k_merkle_scan_place(const ArgLists L, const uint64_t *__restrict__ nodes,
                                                            uint64_t *__restrict__ sa, uint64_t *__restrict__ sb,
                                                            const ArgTables tab, uint64_t ngroups,
                                                            const uint64_t *__restrict__ dirty_mask,
                                                            const SlotBump bump, uint64_t *__restrict__ total,
                                                            uint64_t arena_base)
{
    __shared__ uint64_t lds[4096];  // Merkle values (workgroup 0), then the groups' offsets
    __shared__ uint64_t msk[kScanCompactMaxGroups];
    __shared__ uint64_t lds2[64];
    __shared__ uint64_t roots[kArgBufs];
    __shared__ uint32_t wsum[33];
    static_assert(kScanCompactMaxGroups <= 4 * 1024 && kScanCompactMaxGroups <= 4096,
                  "four dirty masks per thread, offsets in the Merkle LDS array");
    const uint32_t t = threadIdx.x;
    uint64_t mk[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) mk[k] = 4 * t + k < ngroups ? dirty_mask[4 * t + k] : 0;
    const uint64_t top = !bump.bump ? 0 : bump.reset ? bump.reset : *bump.bump;
    if (blockIdx.x == 0) {
        // The masks' round trip to memory overlaps the Merkle reduction.
        merkle_lists<1024>(L, nodes, sa, sb, lds, lds2, roots);
        const uint64_t count = scan_masks_small(mk, ngroups, lds, wsum);
        if (t == 0) *total = count;
        if (t == 1023) place_slots(bump, count, top);
        return;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (4 * t + k < ngroups) msk[4 * t + k] = mk[k];
    const uint64_t count = scan_masks_small(mk, ngroups, lds, wsum);  // ends with a barrier: msk is visible
    const uint32_t lane = t & 63;
    const uint64_t stride = (uint64_t)(gridDim.x - 1) * 16;
    for (uint64_t s = (uint64_t)(blockIdx.x - 1) * 16 + (t >> 6); s < count; s += stride) {
        uint32_t lo = 0, hi = (uint32_t)ngroups;  // lds[lo] <= s (lds[0] = 0)
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) >> 1;
            if (lds[mid] <= s) lo = mid; else hi = mid;
        }
        const uint64_t m = msk[lo];
        const uint32_t k = (uint32_t)(s - lds[lo]);
        const uint32_t below = (uint32_t)__popcll(lane ? m & ((1ULL << lane) - 1) : 0);
        const uint32_t c = (uint32_t)__ffsll((unsigned long long)__ballot(((m >> lane) & 1) && below == k)) - 1;
        const JobBuf &jb = tab.bufs[buf_index(tab, lo)];
        const uint64_t i = (lo - jb.group_begin) * kGroupChunks + c;
        const uint64_t slot_off = top - (s + 1) * kChunk;  // arena offset
        if (lane == 0) ((g_u64 *)jb.manifest)[i] = slot_off;
        copy_chunk(tab, jb, i, arena_base + slot_off, lane);
    }
}

// Slot assignment and dirty copy in one launch (jobs with device tables,
// or whose slots the host placed, after the scan of the dirty masks): one
// wavefront per chunk, four per 256-lane workgroup, striding over the job's
// chunk positions (64 per group) so that a large job launches no more than
// kPlaceBlocks workgroups.  The wavefront of a dirty chunk takes its slot
// (below the payload top in *top_word) from its group's scanned offset and
// the set bits of the mask below it, as k_merkle_scan_place; lane 0 enters the
// slot in the manifest and all 64 lanes copy the chunk into it, 64 bytes per
// lane, zero-padding a partial chunk.  A clean chunk costs its wavefront one
// (cached) mask load: the diff tiles entered it in the manifest.
constexpr uint64_t kPlaceBlocks = 2048;  // 8192 wavefronts: eight workgroups per CU
template <class Tab>
__global__ __launch_bounds__(256) void k_place_dirty(const Tab tab, uint64_t npos, const uint64_t *__restrict__ dirty_mask,
                                                     const uint64_t *__restrict__ offsets,
                                                     const uint64_t *__restrict__ top_word, uint64_t arena_base)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t stride = (uint64_t)gridDim.x * 4;
    for (uint64_t gc = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6); gc < npos; gc += stride) {
        const uint64_t G = gc / kGroupChunks;
        const uint32_t c = (uint32_t)(gc % kGroupChunks);
        const uint64_t mask = dirty_mask[G];
        if (!((mask >> c) & 1)) continue;
        const JobBuf &jb = tab.bufs[buf_index(tab, G)];
        const uint64_t i = (G - jb.group_begin) * kGroupChunks + c;
        if (i >= jb.nchunks) continue;  // (a mask never sets such a bit)
        g_u64 *man = (g_u64 *)jb.manifest;
        const uint64_t slot = offsets[G] + (uint64_t)__popcll(c ? mask & ((1ULL << c) - 1) : 0);
        const uint64_t top = *top_word;  // arena offset
        if (lane == 0) man[i] = top - (slot + 1) * kChunk;
        copy_chunk(tab, jb, i, arena_base + top - (slot + 1) * kChunk, lane);
    }
}

// Copies n slots stored downwards from `top` into increasing order at dst
// (slot s -> dst + s*4096): the readable form of an incremental payload.
__global__ __launch_bounds__(256) void k_reverse_slots(uint64_t top, uint64_t dst, uint64_t n)
{
    const uint64_t s = blockIdx.x;
    if (s >= n) return;
    const uint32_t x = threadIdx.x * 16;
    store16(dst + s * kChunk + x, load16(top - (s + 1) * kChunk + x));
}

// ---------------------------------------------------------------- classify

// Bitmap word G (= one 64-chunk group of one buffer), computed by one
// wavefront: chunk i differs iff its K replay fingerprints are not all equal;
// the wave's ballot is the word.
template <class Tab>
__device__ __forceinline__ uint64_t classify_word(const Tab &tab, uint64_t G, uint32_t lane,
                                                  const uint64_t *hashes, uint32_t K, uint64_t total)
{
    const JobBuf &jb = tab.bufs[buf_index(tab, G)];
    const uint64_t i = (G - jb.group_begin) * kGroupChunks + lane;
    bool differs = false;
    if (i < jb.nchunks) {
        const uint64_t idx = jb.chunk_begin + i;
        const uint64_t h0 = hashes[idx];
        for (uint32_t k = 1; k < K; ++k) differs |= hashes[(uint64_t)k * total + idx] != h0;
    }
    return __ballot(differs);
}

// One wavefront per bitmap word.
template <class Tab>
__global__ __launch_bounds__(64) void k_classify(const Tab tab, const uint64_t *__restrict__ hashes, uint32_t K,
                                                 uint64_t total, uint64_t *__restrict__ bitmap)
{
    const uint64_t word = classify_word(tab, blockIdx.x, threadIdx.x, hashes, K, total);
    if (threadIdx.x == 0) bitmap[blockIdx.x] = word;
}

// Per buffer: 1 iff any of its bitmap words is non-zero (one wavefront per
// buffer, lanes striding over the words).
template <class Tab>
__global__ __launch_bounds__(64) void k_labels(const Tab tab, const uint64_t *__restrict__ bitmap,
                                               uint8_t *__restrict__ labels)
{
    const uint32_t b = blockIdx.x;
    const JobBuf &jb = tab.bufs[b];
    const uint64_t nw = (jb.nchunks + kGroupChunks - 1) / kGroupChunks;
    uint64_t any = 0;
    for (uint64_t w = threadIdx.x; w < nw; w += 64) any |= bitmap[jb.group_begin + w];
    const bool set = __ballot(any != 0) != 0;
    if (threadIdx.x == 0) labels[b] = set ? 1 : 0;
}

// Small jobs (tables in the kernel arguments, at most kClassifyFusedGroups
// groups): the bitmap and the labels in one workgroup and one launch.
// Wavefront w computes words w, w + 16, ... (also kept in LDS); after a
// barrier, one wavefront per buffer ORs its words into the buffer's label.
__global__ __launch_bounds__(1024) void k_classify_small(const ArgTables tab, uint64_t ngroups,
                                                         const uint64_t *__restrict__ hashes, uint32_t K,
                                                         uint64_t total, uint64_t *__restrict__ bitmap,
                                                         uint8_t *__restrict__ labels)
{
    __shared__ uint64_t words[kClassifyFusedGroups];
    const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (uint64_t G = wave; G < ngroups; G += 16) {
        const uint64_t word = classify_word(tab, G, lane, hashes, K, total);
        if (lane == 0) {
            bitmap[G] = word;
            words[G] = word;
        }
    }
    __syncthreads();
    for (uint32_t b = wave; b < tab.nbuf; b += 16) {
        const JobBuf &jb = tab.bufs[b];
        const uint64_t nw = (jb.nchunks + kGroupChunks - 1) / kGroupChunks;
        uint64_t any = 0;
        for (uint64_t w = lane; w < nw; w += 64) any |= words[jb.group_begin + w];
        const bool set = __ballot(any != 0) != 0;
        if (lane == 0) labels[b] = set ? 1 : 0;
    }
}

// Workgroup sizes (lanes) and slice bytes of the tile kernels, from
// measurement on MI355X.
constexpr int kPackLanes = 1024, kPackSlice = 512;
// The staggered verified restore (jobs of 2-9 rounds) moves 1 KiB slices:
// 2-4% faster there than 512 B (the KV ring window 187 -> 182 us, flat
// 128-576 MiB within -4% .. +2%), while the staggered pack is 1-3% slower
// with them and keeps 512 B.
constexpr int kVerifyStaggerSlice = 1024;
// The fused pack of a job of at most this many rounds (one workgroup per CU)
// stores the snapshot through the caches (plain stores), a larger job past
// them (nontemporal stores).  Measured on MI355X in one process, alternating,
// with the loads nontemporal in both: pack + fingerprint of flat 64-127 MiB
// 15-21% faster, 128-576 MiB 3-10%, KV ring windows of 64-576 MiB 4-20%, and
// a checkpoint followed by a restore of it 3-17% faster per step (the
// restore also finds part of the snapshot still in the caches); the 512 MiB
// KV ring step (checkpoint, fork, two restores) 564 -> 551 us.  Above the
// bound write-back stops paying: the 1024-session batch 10.84 -> 11.40 ms
// and flat 1-4 GiB 3-4% slower in the same process.  Restores keep
// nontemporal stores whatever the size (plain ones: the KV ring restore 177
// -> 196 us, its verified restore 181 -> 196 us).
constexpr uint32_t kPackWriteBackMaxRounds = kStaggerMaxRounds;
constexpr int kHashLanes = 256, kHashSlice = 512;
constexpr int kCopyLanes = 512, kCopySlice = 1024;
// Fingerprint and diff tiles of jobs whose tables travel in the kernel
// arguments take 1024 lanes up to a few rounds of groups: one workgroup per
// CU then keeps the whole CU's loads in flight, where 256-lane tiles leave
// part of a round's CUs with one tile and others with two (measured:
// incremental checkpoints of flat 64-512 MiB 4-9% faster, the growing bank's
// late steps 8%; fingerprints of flat 64-256 MiB 8-15%).  With device tables
// a tile's first access is a dependent load of its group-map entry, which
// four 256-lane tiles per CU hide and one 1024-lane tile does not (a wrapping
// KV ring window: diff 115 -> 131 us, fingerprint 89 -> 106 us), so those
// keep 256 lanes.  Above the bounds the wide tiles stop paying: a diff of
// 4096 groups is even and one of 8192 groups 19% slower; a fingerprint of
// 2048 groups is 5% faster on a flat buffer and 1.5% slower on a 64-run KV
// ring window.
constexpr uint64_t kWideDiffGroups = 2048, kWideHashGroups = 1024;
constexpr int kSmallLanes = 256;  // sub-tiles of small jobs: 8 chunks per workgroup
// A sub-tile moves whole chunks in one step (8 granules per lane): a small
// job's time is a tile's latency, one load round trip per step.
constexpr int kSmallSlice = 4096;

// ---------------------------------------------------------------- bank shrink

// Total order on float32 relevance scores as unsigned keys: negative values
// reversed below the positive ones (-0.0 just below +0.0), every NaN above
// +inf.
__device__ __forceinline__ uint32_t score_key(uint32_t bits)
{
    if ((bits & 0x7F800000u) == 0x7F800000u && (bits & 0x007FFFFFu)) return 0xFFFFFFFFu;
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

// hist[b] += 1 for every lane of the wavefront with m set.  AGG: lanes that
// share the first such lane's bucket are added with one atomic (ties, the
// common conflict, cost one LDS atomic per wavefront, not 64 serialised
// ones); worth its extra steps on long streams only.
template <bool AGG>
__device__ __forceinline__ void hist_add(uint32_t *hist, uint32_t b, bool m)
{
    if constexpr (!AGG) {
        if (m) atomicAdd(&hist[b], 1u);
        return;
    }
    const uint64_t act = __ballot(m);
    if (!act) return;
    const int leader = __builtin_ctzll(act);
    const uint32_t lb = (uint32_t)__builtin_amdgcn_readlane((int)b, leader);
    const bool same = m && b == lb;
    const uint64_t sm = __ballot(same);
    if ((int)(threadIdx.x & 63) == leader) atomicAdd(&hist[lb], (uint32_t)__popcll(sm));
    else if (m && !same) atomicAdd(&hist[b], 1u);
}

// Set bits of a wavefront mask in the lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// How a selection reads its n scores.  The array starts head = (address mod
// 16) / 4 scores past a 16-byte boundary; in the aligned view that starts
// there (group g = scores 4g - head .. 4g - head + 3), the whole groups
// [gf0, gf1) are read 16 bytes at a time, and the at most three scores before
// them, [0, e_lo), and after them, [e_hi, n), one at a time.
struct SelView {
    uint64_t base;  // address of score -head (16-byte aligned)
    uint64_t gf0, gf1, e_lo, e_hi;
    uint32_t head;
};
__device__ __forceinline__ SelView sel_view(uint64_t scores, uint32_t n)
{
    SelView v;
    v.head = (uint32_t)(scores & 15) / 4;
    v.base = scores - 4 * v.head;
    v.gf0 = v.head ? 1 : 0;
    const uint64_t g1 = ((uint64_t)n + v.head) / 4;
    v.gf1 = g1 > v.gf0 ? g1 : v.gf0;
    v.e_lo = umin(n, 4 * v.gf0 - v.head);
    const uint64_t hi = umin(n, 4 * v.gf1 - v.head);
    v.e_hi = hi > v.e_lo ? hi : v.e_lo;
    return v;
}
// Keys of U groups: group g0 + stride * u for u < U, or group end - 1 where
// that lies at or past `end` (ok[u] false; a valid address, its keys unused).  All U loads are issued before
// any key is formed (a scheduling barrier keeps the compiler from moving each
// load down to its first use, which would wait on them one at a time).
template <int U>
__device__ __forceinline__ void load_keys(const SelView &v, uint64_t g0, uint64_t stride, uint64_t end,
                                          uint32_t (&k)[U][4], bool (&ok)[U])
{
    v4u32 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint64_t g = g0 + stride * u;
        ok[u] = g < end;
        x[u] = *(const g_v4u32 *)(v.base + 16 * (ok[u] ? g : end - 1));
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j) k[u][j] = score_key(x[u][j]);
}
// Key of score i, read alone.
__device__ __forceinline__ uint32_t key_at(uint64_t scores, uint64_t i) { return score_key(((const g_u32 *)scores)[i]); }

// The single scores a selection reads one at a time (before and after the
// whole groups), one per lane of wavefront 0: lane l < 8 holds score l of
// [0, e_lo) ++ [e_hi, n).  `raw` is loaded at once; its key is formed later,
// so that the load overlaps others.
struct SelSingle {
    uint64_t i;
    bool in, head, tail;
    uint32_t raw;
};
__device__ __forceinline__ SelSingle sel_single(const SelView &v, uint64_t scores, uint32_t n, uint32_t lane,
                                                bool wave0)
{
    SelSingle s;
    s.i = lane < v.e_lo ? lane : v.e_hi + (lane - v.e_lo);
    s.in = wave0 && lane < 8 && s.i < n && (lane < v.e_lo || s.i >= v.e_hi);
    s.head = s.in && lane < v.e_lo;
    s.tail = s.in && lane >= v.e_lo;
    s.raw = 0;
    if (s.in) s.raw = ((const g_u32 *)scores)[s.i];
    return s;
}

// One radix-select pass's choice, in wavefront 0: lane l holds buckets
// 4l..4l+3 of the histogram, and the bucket where the running count first
// reaches `need` is the one.  True in the one lane that finds it, with the
// bucket and the rank of the keep-th key among that bucket's keys.
__device__ __forceinline__ bool pick_bucket(const uint32_t *hist, uint32_t need, uint32_t lane, uint32_t &bucket,
                                            uint32_t &rest)
{
    const uint32_t h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2], h3 = hist[4 * lane + 3];
    const uint32_t sum = h0 + h1 + h2 + h3;
    const uint32_t incl = wave_incl_scan(sum);
    uint32_t cum = incl - sum;
    if (!(cum < need && incl >= need)) return false;
    uint32_t d = 4 * lane;
    if (cum + h0 < need) {
        cum += h0;
        ++d;
        if (cum + h1 < need) {
            cum += h1;
            ++d;
            if (cum + h2 < need) {
                cum += h2;
                ++d;
            }
        }
    }
    bucket = d;
    rest = need - cum;
    return true;
}

// Counts of keys below and equal to K* among the single scores (head pair,
// tail pair); every lane of wavefront 0 gets them.
__device__ __forceinline__ void count_singles(const SelSingle &s, uint32_t key, uint32_t prefix, uint32_t (&c)[4])
{
    c[0] = (uint32_t)__popcll(__ballot(s.head && key < prefix));
    c[1] = (uint32_t)__popcll(__ballot(s.head && key == prefix));
    c[2] = (uint32_t)__popcll(__ballot(s.tail && key < prefix));
    c[3] = (uint32_t)__popcll(__ballot(s.tail && key == prefix));
}

// Writes the kept single scores, wavefront 0: lane order is index order
// within the head and the tail; (ph, rh) and (pt, rt) are the kept entries
// and K* keys before each.
__device__ __forceinline__ void place_singles(const SelSingle &s, uint32_t key, uint32_t prefix, uint32_t need,
                                              uint32_t ph, uint32_t rh, uint32_t pt, uint32_t rt,
                                              uint32_t *__restrict__ kept)
{
    const uint64_t eqh = __ballot(s.head && key == prefix), eqt = __ballot(s.tail && key == prefix);
    const uint32_t r = s.head ? rh + lanes_below(eqh) : rt + lanes_below(eqt);
    const bool take = s.in && (key < prefix || (key == prefix && r < need));
    const uint64_t th = __ballot(s.head && take), tt = __ballot(s.tail && take);
    if (take) kept[s.head ? ph + lanes_below(th) : pt + lanes_below(tt)] = (uint32_t)s.i;
}

// Writes the kept indices of one whole group per lane of a wavefront, in
// index order (lane by lane, score by score); every lane takes part
// (ballots).  The K* keys and kept entries before score j of a lane: those
// of the lanes below, then its own before j.  pos and rank (kept entries and
// K* keys before this wavefront's groups) advance, the same in every lane.
__device__ __forceinline__ void place_group(const uint32_t (&k)[4], bool ok, uint64_t g, uint32_t head,
                                            uint32_t prefix, uint32_t need, uint32_t &pos, uint32_t &rank,
                                            uint32_t *__restrict__ kept)
{
    uint64_t em[4], tm[4];
    uint32_t r = rank, take = 0, o = pos;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        em[j] = __ballot(ok && k[j] == prefix);
        r += lanes_below(em[j]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (!ok) continue;
        if (k[j] < prefix) take |= 1u << j;
        else if (k[j] == prefix && r++ < need) take |= 1u << j;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        tm[j] = __ballot((take >> j) & 1);
        o += lanes_below(tm[j]);
    }
    const uint64_t e0 = 4 * g - head;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if ((take >> j) & 1) kept[o++] = (uint32_t)(e0 + j);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        rank += (uint32_t)__popcll(em[j]);
        pos += (uint32_t)__popcll(tm[j]);
    }
}

// Selection of a bank of at most kSelectOneWorkgroupEntries scores in one
// workgroup of 1024 lanes: the `keep` best-ranked entries (a smaller key, or
// an equal key at a lower index, ranks first) in increasing index order.
//   1. Radix select, most significant byte first: four passes histogram the
//      candidates' next byte (LDS atomics) and narrow to the bucket that holds
//      the keep-th smallest key (wavefront 0 finds it with a prefix sum over
//      the 256 buckets), which ends as K*, with `need` = how many entries
//      with key K* are kept (those with the lowest indices).
//   2. Sixteen ranges of a multiple of 64 whole groups, one per wavefront
//      (up to 1024 groups each lane holds its one group, read once for every
//      pass), count their keys below K* and equal to K*; the counts of the ranges before a range give the rank
//      of its first K* key, hence how many entries it keeps, and where its
//      kept indices go.  The single scores before and after the whole groups
//      are ranges of their own, first and last, held by wavefront 0.
//   3. Each wavefront compacts its kept indices with ballots.
// Larger banks take the multi-workgroup selection (k_sel_*), which follows
// the same steps with a launch per pass.
// Up to here one workgroup is faster (26 us at 16384 scores, 45 us at 32768)
// than the twelve launches of the multi-workgroup selection (55 us at 16385
// to 65536, 69 us at 2^20, 1.7 ms at 2^28 where one workgroup took 330 ms).
constexpr uint32_t kSelectOneWorkgroupEntries = 32768;
__global__ __launch_bounds__(1024) void k_shrink_select(uint64_t scores, uint32_t n, uint32_t keep,
                                                        uint32_t *__restrict__ kept)
{
    // Per range: keys below K* (cnt[r]) and equal to K* (cnt[18 + r]); range 0
    // = the single scores before the whole groups, 1 + w = wavefront w's
    // groups, 17 = the single scores after.
    __shared__ uint32_t hist[256];
    __shared__ uint32_t cnt[36];
    __shared__ uint32_t pick[2];
    const uint32_t t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const SelView v = sel_view(scores, n);
    const uint64_t nfull = v.gf1 - v.gf0, per = (nfull + 1023) / 1024 * 64;
    const uint64_t w0 = v.gf0 + umin(wave * per, nfull), w1 = v.gf0 + umin(wave * per + per, nfull);
    const bool resident = nfull <= 1024;  // each lane holds its one group for every pass
    const SelSingle es = sel_single(v, scores, n, lane, wave == 0);
    uint32_t rk[1][4] = {{0, 0, 0, 0}};
    bool rok[1] = {false};
    if (resident && w0 < w1) load_keys<1>(v, w0 + lane, 64, w1, rk, rok);
    const uint32_t ek = score_key(es.raw);

    uint32_t prefix = 0, pmask = 0, need = keep;  // need: 1-based rank of K* among the candidates
    for (int p = 0; p < 4; ++p) {
        const uint32_t shift = 24 - 8 * p;
        if (t < 256) hist[t] = 0;
        __syncthreads();
        if (resident) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                hist_add<false>(hist, (rk[0][j] >> shift) & 255u, rok[0] && (rk[0][j] & pmask) == prefix);
        } else {
            for (uint64_t g0 = w0; g0 < w1; g0 += 64) {
                uint32_t k[1][4];
                bool ok[1];
                load_keys<1>(v, g0 + lane, 64, w1, k, ok);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    hist_add<false>(hist, (k[0][j] >> shift) & 255u, ok[0] && (k[0][j] & pmask) == prefix);
            }
        }
        if (wave == 0) hist_add<false>(hist, (ek >> shift) & 255u, es.in && (ek & pmask) == prefix);
        __syncthreads();
        uint32_t bucket, rest;
        if (t < 64 && pick_bucket(hist, need, lane, bucket, rest)) {
            pick[0] = bucket;
            pick[1] = rest;
        }
        __syncthreads();
        prefix |= pick[0] << shift;
        pmask |= 255u << shift;
        need = pick[1];
        __syncthreads();
    }

    // 2. Counts per range (wavefront totals, the same in every lane).
    uint32_t lt = 0, eq = 0;
    const auto count = [&](const uint32_t(&k)[4], bool ok) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            lt += (uint32_t)__popcll(__ballot(ok && k[j] < prefix));
            eq += (uint32_t)__popcll(__ballot(ok && k[j] == prefix));
        }
    };
    if (resident) {
        count(rk[0], rok[0]);
    } else {
        for (uint64_t g0 = w0; g0 < w1; g0 += 64) {
            uint32_t k[1][4];
            bool ok[1];
            load_keys<1>(v, g0 + lane, 64, w1, k, ok);
            count(k[0], ok[0]);
        }
    }
    if (lane == 0) {
        cnt[1 + wave] = lt;
        cnt[19 + wave] = eq;
    }
    if (wave == 0) {
        uint32_t c[4];
        count_singles(es, ek, prefix, c);
        if (lane == 0) {
            cnt[0] = c[0];
            cnt[18] = c[1];
            cnt[17] = c[2];
            cnt[35] = c[3];
        }
    }
    __syncthreads();

    // 3. Placement.  Kept entries (pos) and K* keys (rank) in the ranges
    // before range r:
    const auto range_start = [&](uint32_t r, uint32_t &pos, uint32_t &rank) {
        pos = rank = 0;
        for (uint32_t x = 0; x < r; ++x) {
            const uint32_t e = cnt[18 + x];
            pos += cnt[x] + (need > rank ? min(need - rank, e) : 0u);
            rank += e;
        }
    };
    if (wave == 0) {
        uint32_t ph, rh, pt, rt;
        range_start(0, ph, rh);
        range_start(17, pt, rt);
        place_singles(es, ek, prefix, need, ph, rh, pt, rt, kept);
    }
    uint32_t pos, rank;
    range_start(1 + wave, pos, rank);
    const uint32_t pos_end = pos + lt + (need > rank ? min(need - rank, eq) : 0u);
    if (resident) {
        if (pos < pos_end) place_group(rk[0], rok[0], w0 + lane, v.head, prefix, need, pos, rank, kept);
    } else {
        for (uint64_t g0 = w0; g0 < w1 && pos < pos_end; g0 += 64) {
            uint32_t k[1][4];
            bool ok[1];
            load_keys<1>(v, g0 + lane, 64, w1, k, ok);
            place_group(k[0], ok[0], g0 + lane, v.head, prefix, need, pos, rank, kept);
        }
    }
}

// ---- multi-workgroup selection (banks of more than kSelectOneWorkgroupEntries
// scores).  The same steps as k_shrink_select, a launch each: k_sel_init,
// then per radix pass k_sel_hist (every workgroup adds its LDS histogram
// into the pass's device histogram) and k_sel_pick (one wavefront narrows the
// prefix), then k_sel_count (keys below / equal to K* per wavefront range),
// k_sel_scan (where each range's kept indices go) and k_sel_place.  The
// whole groups are cut into one range of a multiple of 64 groups per
// wavefront of the grid, read with 8 groups per lane in flight; range 0 and
// range R - 1 are the single scores, held by wavefront 0 of workgroup 0.
struct SelState {
    uint32_t prefix, pmask, need, pad;
    uint32_t hist[2][256];  // pass p adds into hist[p % 2]; pick p clears the other
};
constexpr int kSelU = 8;
__device__ __forceinline__ void sel_wave_range(const SelView &v, uint64_t gw, uint64_t nwaves, uint64_t &w0,
                                               uint64_t &w1)
{
    const uint64_t nfull = v.gf1 - v.gf0;
    const uint64_t per = (nfull + 64 * nwaves - 1) / (64 * nwaves) * 64;
    w0 = v.gf0 + umin(gw * per, nfull);
    w1 = v.gf0 + umin(gw * per + per, nfull);
}

__global__ __launch_bounds__(256) void k_sel_init(SelState *__restrict__ st, uint32_t keep)
{
    if (threadIdx.x == 0) {
        st->prefix = 0;
        st->pmask = 0;
        st->need = keep;
    }
    st->hist[0][threadIdx.x] = 0;
}

__global__ __launch_bounds__(1024) void k_sel_hist(uint64_t scores, uint32_t n, SelState *__restrict__ st, int p)
{
    __shared__ uint32_t hist[256];
    const uint32_t t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const SelView v = sel_view(scores, n);
    const uint32_t shift = 24 - 8 * p, prefix = st->prefix, pmask = st->pmask;
    if (t < 256) hist[t] = 0;
    __syncthreads();
    uint64_t w0, w1;
    sel_wave_range(v, (uint64_t)blockIdx.x * 16 + wave, (uint64_t)gridDim.x * 16, w0, w1);
    for (uint64_t g0 = w0; g0 < w1; g0 += 64ull * kSelU) {
        uint32_t k[kSelU][4];
        bool ok[kSelU];
        load_keys<kSelU>(v, g0 + lane, 64, w1, k, ok);
#pragma unroll
        for (int u = 0; u < kSelU; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                hist_add<true>(hist, (k[u][j] >> shift) & 255u, ok[u] && (k[u][j] & pmask) == prefix);
    }
    if (blockIdx.x == 0 && wave == 0) {
        const SelSingle es = sel_single(v, scores, n, lane, true);
        const uint32_t ek = score_key(es.raw);
        hist_add<true>(hist, (ek >> shift) & 255u, es.in && (ek & pmask) == prefix);
    }
    __syncthreads();
    if (t < 256 && hist[t]) atomicAdd(&st->hist[p & 1][t], hist[t]);
}

__global__ __launch_bounds__(64) void k_sel_pick(SelState *__restrict__ st, int p)
{
    const uint32_t lane = threadIdx.x, shift = 24 - 8 * p;
    uint32_t bucket, rest;
    if (pick_bucket(st->hist[p & 1], st->need, lane, bucket, rest)) {
        st->prefix |= bucket << shift;
        st->pmask |= 255u << shift;
        st->need = rest;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) st->hist[(p + 1) & 1][4 * lane + i] = 0;
}

// Range r's keys below K* (lt[r]) and equal to K* (eq[r]).
__global__ __launch_bounds__(1024) void k_sel_count(uint64_t scores, uint32_t n, const SelState *__restrict__ st,
                                                    uint32_t *__restrict__ lt_out, uint32_t *__restrict__ eq_out)
{
    const uint32_t t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const SelView v = sel_view(scores, n);
    const uint32_t prefix = st->prefix;
    const uint64_t gw = (uint64_t)blockIdx.x * 16 + wave, nwaves = (uint64_t)gridDim.x * 16;
    uint64_t w0, w1;
    sel_wave_range(v, gw, nwaves, w0, w1);
    uint32_t lt = 0, eq = 0;
    for (uint64_t g0 = w0; g0 < w1; g0 += 64ull * kSelU) {
        uint32_t k[kSelU][4];
        bool ok[kSelU];
        load_keys<kSelU>(v, g0 + lane, 64, w1, k, ok);
#pragma unroll
        for (int u = 0; u < kSelU; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                lt += (uint32_t)__popcll(__ballot(ok[u] && k[u][j] < prefix));
                eq += (uint32_t)__popcll(__ballot(ok[u] && k[u][j] == prefix));
            }
    }
    if (lane == 0) {
        lt_out[1 + gw] = lt;
        eq_out[1 + gw] = eq;
    }
    if (blockIdx.x == 0 && wave == 0) {
        const SelSingle es = sel_single(v, scores, n, lane, true);
        uint32_t c[4];
        count_singles(es, score_key(es.raw), prefix, c);
        if (lane == 0) {
            lt_out[0] = c[0];
            eq_out[0] = c[1];
            lt_out[nwaves + 1] = c[2];
            eq_out[nwaves + 1] = c[3];
        }
    }
}

// Where each of the R ranges starts: the kept entries before it (pos) are
// the keys below K* before it plus the first `need` K* keys, so pos =
// LT + min(need, EQ) and rank = EQ for the exclusive prefix sums LT and EQ of
// the counts.  One workgroup; every thread scans a contiguous segment.
__global__ __launch_bounds__(1024) void k_sel_scan(const SelState *__restrict__ st, const uint32_t *__restrict__ lt,
                                                   const uint32_t *__restrict__ eq, uint32_t R,
                                                   uint32_t *__restrict__ pos_out, uint32_t *__restrict__ rank_out)
{
    __shared__ uint32_t wsum[2][33];
    const uint32_t t = threadIdx.x, wave = t >> 6, lane = t & 63;
    const uint32_t per = (R + 1023) / 1024, s0 = min(t * per, R), s1 = min(s0 + per, R);
    uint32_t a = 0, b = 0;
    for (uint32_t r = s0; r < s1; ++r) {
        a += lt[r];
        b += eq[r];
    }
    const uint32_t ia = wave_incl_scan(a), ib = wave_incl_scan(b);
    if (lane == 63) {
        wsum[0][wave] = ia;
        wsum[1][wave] = ib;
    }
    __syncthreads();
    if (wave == 0) {
        const uint32_t x = lane < 16 ? wsum[0][lane] : 0, y = lane < 16 ? wsum[1][lane] : 0;
        const uint32_t xi = wave_incl_scan(x), yi = wave_incl_scan(y);
        if (lane < 16) {
            wsum[0][16 + lane] = xi - x;
            wsum[1][16 + lane] = yi - y;
        }
    }
    __syncthreads();
    const uint32_t need = st->need;
    uint32_t LT = ia - a + wsum[0][16 + wave], EQ = ib - b + wsum[1][16 + wave];
    for (uint32_t r = s0; r < s1; ++r) {
        pos_out[r] = LT + min(need, EQ);
        rank_out[r] = EQ;
        LT += lt[r];
        EQ += eq[r];
    }
}

__global__ __launch_bounds__(1024) void k_sel_place(uint64_t scores, uint32_t n, const SelState *__restrict__ st,
                                                    const uint32_t *__restrict__ pos_in,
                                                    const uint32_t *__restrict__ rank_in, uint32_t *__restrict__ kept)
{
    const uint32_t t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const SelView v = sel_view(scores, n);
    const uint32_t prefix = st->prefix, need = st->need;
    const uint64_t gw = (uint64_t)blockIdx.x * 16 + wave, nwaves = (uint64_t)gridDim.x * 16;
    if (blockIdx.x == 0 && wave == 0) {
        const SelSingle es = sel_single(v, scores, n, lane, true);
        place_singles(es, score_key(es.raw), prefix, need, pos_in[0], rank_in[0], pos_in[nwaves + 1],
                      rank_in[nwaves + 1], kept);
    }
    uint64_t w0, w1;
    sel_wave_range(v, gw, nwaves, w0, w1);
    uint32_t pos = pos_in[1 + gw], rank = rank_in[1 + gw];
    const uint32_t pos_end = pos_in[2 + gw];  // the next range's start
    for (uint64_t g0 = w0; g0 < w1 && pos < pos_end; g0 += 64ull * kSelU) {
        uint32_t k[kSelU][4];
        bool ok[kSelU];
        load_keys<kSelU>(v, g0 + lane, 64, w1, k, ok);
#pragma unroll
        for (int u = 0; u < kSelU; ++u) place_group(k[u], ok[u], g0 + 64ull * u + lane, v.head, prefix, need, pos, rank, kept);
    }
}

// Moves of a bank shrink, every part in one launch; work item w is slice sl
// of kept entry j of the part whose items hold w (the part is the same for
// all lanes of a workgroup).  Kept indices increase, so kept[j] >= j, and in
// place the entries overwritten are the destinations j < keep.  A source
// kept[j] < keep (other than j itself) is such a destination, written by
// another item of the same pass: STAGE copies those sources to the part's
// staging area (slot j) first.  The place pass then writes destination j
// from the staging area, or straight from a source kept[j] >= keep, which no
// destination overwrites, and in place skips kept[j] == j (already there).
// Out-of-place parts gather straight from the source and do nothing in the
// stage pass.
__device__ __forceinline__ void move_granule(uint64_t a, uint64_t d, uint64_t g)
{
    if (g == 16) store16_nt(d, load16_nt(a));
    else if (g == 4) *(g_u32 *)d = *(const g_u32 *)a;
    else *(g_u8 *)d = *(const g_u8 *)a;
}
template <bool STAGE>
__global__ __launch_bounds__(256) void k_move_entries(const ShrinkParts P, const uint32_t *__restrict__ kept,
                                                      uint64_t keep)
{
    for (uint64_t w = blockIdx.x; w < P.items; w += gridDim.x) {
        uint32_t p = 0;
        while (p + 1 < P.n && P.p[p + 1].item_begin <= w) ++p;
        const ShrinkPart &q = P.p[p];
        const uint64_t r = w - q.item_begin, j = r / q.spe, x = ((r % q.spe) * 256 + threadIdx.x) * q.g;
        if (x >= q.eb) continue;
        const uint64_t e = kept[j];
        const bool in_place = q.stage != 0;
        if (STAGE) {
            if (in_place && e < keep && e != j) move_granule(q.src + e * q.eb + x, q.stage + j * q.eb + x, q.g);
        } else if (!(in_place && e == j)) {
            const uint64_t a = in_place && e < keep ? q.stage + j * q.eb : q.src + e * q.eb;
            move_granule(a + x, q.dst + j * q.eb + x, q.g);
        }
    }
}

// Flips the lowest bit of one byte (the control of the discovery procedure
// gives a component a wrong value this way).
__global__ void k_flip_bit(uint64_t addr)
{
    if (threadIdx.x == 0) *(g_u8 *)addr ^= 1;
}

}  // namespace

// ---------------------------------------------------------------- launchers

hipError_t launch_group_map(const JobBuf *bufs, const Run *runs, uint32_t nbuf, uint64_t ngroups, GroupRef *map,
                            hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((ngroups + 255) / 256);
    run_kernel(k_group_map, dim3(blocks), dim3(256), s, bufs, runs, nbuf, ngroups, map);
    return hipGetLastError();
}

template <class Tab>
hipError_t launch_tile(const Tab &tab, uint64_t ngroups, int mode, uint64_t *nodes, uint64_t *flag_mask,
                       uint64_t arena_base, hipStream_t s, uint32_t tiles_per_group, TileDevice dev)
{
    if (ngroups == 0) return hipSuccess;
    const bool split = tiles_per_group != 1;
    if (split && (mode != kModeHash && mode != kModePack && mode != kModeDiff)) return hipErrorInvalidValue;
    Stagger stg{0, 0};
    if (!split && (mode == kModePack || mode == kModeVerify) && dev.cus && dev.wall_khz &&
        ngroups >= (uint64_t)kStaggerMinRounds * dev.cus && ngroups <= (uint64_t)kStaggerMaxRounds * dev.cus)
        stg = Stagger{dev.cus, (uint32_t)((uint64_t)kStaggerPhaseNs * dev.wall_khz / 1000000)};
    const dim3 grid((uint32_t)(ngroups * tiles_per_group));
    if (tiles_per_group == kSmallTiles) {
        constexpr int kCPW = kGroupChunks / kSmallTiles;
        static_assert(kCPW == 8, "a diff sub-tile writes one mask byte");
        if (mode == kModeHash)
            run_kernel((k_hash<Tab, kModeHash, kSmallLanes, kSmallSlice, kCPW, false>), grid, dim3(kSmallLanes), s,
                       tab, nodes, flag_mask, arena_base);
        else if (mode == kModePack)  // sub-tile jobs are far within the write-back bound
            run_kernel((k_hash<Tab, kModePack, kSmallLanes, kSmallSlice, kCPW, true>), grid, dim3(kSmallLanes), s, tab,
                       nodes, flag_mask, arena_base);
        else
            run_kernel((k_hash<Tab, kModeDiff, kSmallLanes, kSmallSlice, kCPW, false>), grid, dim3(kSmallLanes), s,
                       tab, nodes, flag_mask, arena_base);
        return hipGetLastError();
    }
    if (split) return hipErrorInvalidValue;
    constexpr bool kArgTab = std::is_same<Tab, ArgTables>::value;
    switch (mode) {
    case kModeHash:
        if (kArgTab && ngroups <= kWideHashGroups)
            run_kernel((k_hash<Tab, kModeHash, kPackLanes, kHashSlice, kGroupChunks, false>), grid, dim3(kPackLanes), s,
                       tab, nodes, flag_mask, arena_base);
        else
            run_kernel((k_hash<Tab, kModeHash, kHashLanes, kHashSlice, kGroupChunks, false>), grid, dim3(kHashLanes), s,
                       tab, nodes, flag_mask, arena_base);
        break;
    case kModePack:
        if (stg.ticks)
            run_kernel((k_hash_staggered<Tab, kModePack, kPackLanes, kPackSlice, kGroupChunks>), grid, dim3(kPackLanes),
                       s, tab, nodes, flag_mask, arena_base, stg);
        else if (ngroups <= (uint64_t)kPackWriteBackMaxRounds * std::max<uint32_t>(dev.cus, 1))
            run_kernel((k_hash<Tab, kModePack, kPackLanes, kPackSlice, kGroupChunks, true>), grid, dim3(kPackLanes), s,
                       tab, nodes, flag_mask, arena_base);
        else
            run_kernel((k_hash<Tab, kModePack, kPackLanes, kPackSlice, kGroupChunks, false>), grid, dim3(kPackLanes), s,
                       tab, nodes, flag_mask, arena_base);
        break;
    case kModeDiff:
        if (kArgTab && ngroups <= kWideDiffGroups)
            run_kernel((k_hash<Tab, kModeDiff, kPackLanes, kHashSlice, kGroupChunks, false>), grid, dim3(kPackLanes), s,
                       tab, nodes, flag_mask, arena_base);
        else
            run_kernel((k_hash<Tab, kModeDiff, kHashLanes, kHashSlice, kGroupChunks, false>), grid, dim3(kHashLanes), s,
                       tab, nodes, flag_mask, arena_base);
        break;
    case kModeVerify:
        if (stg.ticks)
            run_kernel((k_hash_staggered<Tab, kModeVerify, kPackLanes, kVerifyStaggerSlice, kGroupChunks>), grid,
                       dim3(kPackLanes), s, tab, nodes, flag_mask, arena_base, stg);
        else
            run_kernel((k_hash<Tab, kModeVerify, kPackLanes, kPackSlice, kGroupChunks, false>), grid,
                       dim3(kPackLanes), s, tab, nodes, flag_mask, arena_base);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Copies need no per-group output, so a small job is cut into sub-tiles here.
template <class Tab>
hipError_t launch_copy(const Tab &tab, uint64_t ngroups, bool pack, uint64_t arena_base, hipStream_t s, uint32_t cus)
{
    if (ngroups == 0) return hipSuccess;
    const uint32_t tiles = tile_split(ngroups);
    const dim3 grid((uint32_t)(ngroups * tiles));
    const bool wb = pack && ngroups <= (uint64_t)kPackWriteBackMaxRounds * cus;
    if (tiles == kSmallTiles) {
        constexpr int kCPW = kGroupChunks / kSmallTiles;
        if (pack)
            run_kernel((k_copy<Tab, true, kSmallLanes, kSmallSlice, kCPW>), grid, dim3(kSmallLanes), s, tab,
                       arena_base, wb);
        else
            run_kernel((k_copy<Tab, false, kSmallLanes, kSmallSlice, kCPW>), grid, dim3(kSmallLanes), s, tab,
                       arena_base, false);
    } else if (pack) {
        run_kernel((k_copy<Tab, true, kCopyLanes, kCopySlice, kGroupChunks>), grid, dim3(kCopyLanes), s, tab,
                   arena_base, wb);
    } else {
        run_kernel((k_copy<Tab, false, kCopyLanes, kCopySlice, kGroupChunks>), grid, dim3(kCopyLanes), s, tab,
                   arena_base, false);
    }
    return hipGetLastError();
}

template <class Tab>
hipError_t launch_place_dirty(const Tab &tab, uint64_t ngroups, const uint64_t *dirty_mask, const uint64_t *offsets,
                              const uint64_t *top_word, uint64_t arena_base, hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    const uint64_t npos = ngroups * kGroupChunks;
    const uint32_t blocks = (uint32_t)std::min<uint64_t>((npos + 3) / 4, kPlaceBlocks);
    run_kernel((k_place_dirty<Tab>), dim3(blocks), dim3(256), s, tab, npos, dirty_mask, offsets, top_word, arena_base);
    return hipGetLastError();
}

template <class Tab>
hipError_t launch_classify(const Tab &tab, uint64_t ngroups, const uint64_t *hashes, uint32_t K, uint64_t total,
                           uint64_t *bitmap, hipStream_t s)
{
    if (ngroups == 0) return hipSuccess;
    run_kernel((k_classify<Tab>), dim3((uint32_t)ngroups), dim3(64), s, tab, hashes, K, total, bitmap);
    return hipGetLastError();
}

template <class Tab>
hipError_t launch_labels(const Tab &tab, const uint64_t *bitmap, uint8_t *labels, hipStream_t s)
{
    if (tab.nbuf == 0) return hipSuccess;
    run_kernel((k_labels<Tab>), dim3(tab.nbuf), dim3(64), s, tab, bitmap, labels);
    return hipGetLastError();
}

hipError_t launch_classify_small(const ArgTables &tab, uint64_t ngroups, const uint64_t *hashes, uint32_t K,
                                 uint64_t total, uint64_t *bitmap, uint8_t *labels, hipStream_t s)
{
    if (ngroups > kClassifyFusedGroups) return hipErrorInvalidValue;
    if (tab.nbuf == 0) return hipSuccess;
    run_kernel(k_classify_small, dim3(1), dim3(1024), s, tab, ngroups, hashes, K, total, bitmap, labels);
    return hipGetLastError();
}

hipError_t launch_merkle(const MerkleList *lists, uint32_t nlists, const uint64_t *in,
                         uint64_t *scratch_a, uint64_t *scratch_b, uint64_t *roots_out,
                         uint64_t max_count, bool pre, hipStream_t s)
{
    if (nlists == 0) return hipSuccess;
    if (max_count > kMerkleLdsValues)
        run_kernel(k_merkle<1024>, dim3(nlists), dim3(1024), s, lists, in, scratch_a, scratch_b, roots_out, pre);
    else
        run_kernel(k_merkle<256>, dim3(nlists), dim3(256), s, lists, in, scratch_a, scratch_b, roots_out, pre);
    return hipGetLastError();
}

hipError_t launch_merkle_blocks(const LongLists &lists, const uint64_t *in, uint64_t *scratch_a, hipStream_t s)
{
    if (lists.n == 0 || lists.n > kLongLists) return lists.n ? hipErrorInvalidValue : hipSuccess;
    const uint64_t waves = lists.block_begin[lists.n];
    if (waves == 0) return hipSuccess;
    run_kernel(k_merkle_blocks, dim3((uint32_t)((waves + 3) / 4)), dim3(256), s, lists, in, scratch_a);
    return hipGetLastError();
}

hipError_t launch_merkle_small(const ArgLists &lists, const uint64_t *in, uint64_t *scratch_a,
                               uint64_t *scratch_b, bool pre, hipStream_t s)
{
    if (lists.nlists == 0) return hipSuccess;
    run_kernel(k_merkle_small, dim3(1), dim3(1024), s, lists, in, scratch_a, scratch_b, pre);
    return hipGetLastError();
}

hipError_t launch_scan(const uint64_t *dirty_mask, uint64_t n, uint64_t *offsets, uint64_t *total,
                       const SlotBump &bump, hipStream_t s)
{
    run_kernel(k_scan<MaskBits>, dim3(1), dim3(1024), s, MaskBits{dirty_mask}, n, offsets, total, bump);
    return hipGetLastError();
}

hipError_t launch_merkle_scan_place(const ArgLists &lists, const uint64_t *nodes, uint64_t *scratch_a,
                                    uint64_t *scratch_b, const ArgTables &tab, uint64_t ngroups,
                                    const uint64_t *dirty_mask, const SlotBump &bump, uint64_t *total,
                                    uint64_t arena_base, hipStream_t s)
{
    if (ngroups > kScanCompactMaxGroups) return hipErrorInvalidValue;
    if (ngroups && (!bump.bump || !bump.bump_out || bump.bump == bump.bump_out)) return hipErrorInvalidValue;
    // Workgroup 0, then enough 16-wavefront workgroups for one stored chunk
    // per wavefront if every chunk is stored (at most kPlaceBlocks / 4).
    const uint64_t npos = ngroups * kGroupChunks;
    const uint32_t blocks = 1 + (uint32_t)std::min<uint64_t>((npos + 15) / 16, kPlaceBlocks / 4);
    run_kernel(k_merkle_scan_place, dim3(blocks), dim3(1024), s, lists, nodes, scratch_a, scratch_b, tab, ngroups,
               dirty_mask, bump, total, arena_base);
    return hipGetLastError();
}

// Scratch of a multi-workgroup selection: SelState, then lt, eq, pos and
// rank arrays of R = 16 x workgroups + 2 ranges.
constexpr uint32_t kSelBlocks = 2048;
static uint32_t select_blocks(uint32_t n) { return std::max<uint32_t>(1, std::min<uint32_t>((n + 4095) / 4096, kSelBlocks)); }
static uint64_t sel_array_bytes(uint32_t R) { return ((uint64_t)R * 4 + 255) / 256 * 256; }
static uint64_t sel_state_bytes() { return (sizeof(SelState) + 255) / 256 * 256; }

uint32_t select_steps(uint32_t n) { return n > kSelectOneWorkgroupEntries ? 12 : 1; }

uint64_t select_scratch_bytes(uint32_t n)
{
    if (n <= kSelectOneWorkgroupEntries) return 0;
    return sel_state_bytes() + 4 * sel_array_bytes(select_blocks(n) * 16 + 2);
}

hipError_t launch_shrink_select(const float *scores, uint32_t n, uint32_t keep, uint32_t *kept, uint64_t scratch,
                                uint32_t step, hipStream_t s)
{
    if (n == 0 || keep == 0) return hipSuccess;
    if (keep > n || step >= select_steps(n)) return hipErrorInvalidValue;
    if ((uint64_t)scores & 3) return hipErrorInvalidValue;
    const uint64_t sc = (uint64_t)scores;
    if (n <= kSelectOneWorkgroupEntries) {
        run_kernel(k_shrink_select, dim3(1), dim3(1024), s, sc, n, keep, kept);
        return hipGetLastError();
    }
    if (!scratch || (scratch & 255)) return hipErrorInvalidValue;
    const uint32_t B = select_blocks(n), R = B * 16 + 2;
    SelState *st = (SelState *)scratch;
    uint32_t *lt = (uint32_t *)(scratch + sel_state_bytes());
    uint32_t *eq = (uint32_t *)((uint64_t)lt + sel_array_bytes(R));
    uint32_t *pos = (uint32_t *)((uint64_t)eq + sel_array_bytes(R));
    uint32_t *rank = (uint32_t *)((uint64_t)pos + sel_array_bytes(R));
    if (step == 0) {
        run_kernel(k_sel_init, dim3(1), dim3(256), s, st, keep);
    } else if (step <= 8) {
        const int p = (int)(step - 1) / 2;
        if (step % 2) run_kernel(k_sel_hist, dim3(B), dim3(1024), s, sc, n, st, p);
        else run_kernel(k_sel_pick, dim3(1), dim3(64), s, st, p);
    } else if (step == 9) {
        run_kernel(k_sel_count, dim3(B), dim3(1024), s, sc, n, (const SelState *)st, lt, eq);
    } else if (step == 10) {
        run_kernel(k_sel_scan, dim3(1), dim3(1024), s, (const SelState *)st, (const uint32_t *)lt,
                   (const uint32_t *)eq, R, pos, rank);
    } else {
        run_kernel(k_sel_place, dim3(B), dim3(1024), s, sc, n, (const SelState *)st, (const uint32_t *)pos,
                   (const uint32_t *)rank, kept);
    }
    return hipGetLastError();
}

hipError_t launch_move_entries(const ShrinkParts &parts, const uint32_t *kept, uint64_t keep, bool stage,
                               hipStream_t s)
{
    if (parts.n > kShrinkParts) return hipErrorInvalidValue;
    if (parts.items == 0) return hipSuccess;
    const uint32_t grid = (uint32_t)std::min<uint64_t>(parts.items, 1u << 20);
    if (stage) run_kernel(k_move_entries<true>, dim3(grid), dim3(256), s, parts, kept, keep);
    else run_kernel(k_move_entries<false>, dim3(grid), dim3(256), s, parts, kept, keep);
    return hipGetLastError();
}

hipError_t launch_flip_bit(uint64_t addr, hipStream_t s)
{
    run_kernel(k_flip_bit, dim3(1), dim3(64), s, addr);
    return hipGetLastError();
}

hipError_t launch_reverse_slots(uint64_t top, uint64_t dst, uint64_t n, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    run_kernel(k_reverse_slots, dim3((uint32_t)n), dim3(256), s, top, dst, n);
    return hipGetLastError();
}

#define PCS_INSTANTIATE(Tab)                                                                                        \
    template hipError_t launch_tile<Tab>(const Tab &, uint64_t, int, uint64_t *, uint64_t *, uint64_t, hipStream_t, \
                                         uint32_t, TileDevice);                                                   \
    template hipError_t launch_copy<Tab>(const Tab &, uint64_t, bool, uint64_t, hipStream_t, uint32_t);           \
    template hipError_t launch_place_dirty<Tab>(const Tab &, uint64_t, const uint64_t *, const uint64_t *,        \
                                                const uint64_t *, uint64_t, hipStream_t);                         \
    template hipError_t launch_classify<Tab>(const Tab &, uint64_t, const uint64_t *, uint32_t, uint64_t,         \
                                             uint64_t *, hipStream_t);                                            \
    template hipError_t launch_labels<Tab>(const Tab &, const uint64_t *, uint8_t *, hipStream_t);
PCS_INSTANTIATE(DevTables)
PCS_INSTANTIATE(ArgTables)
#undef PCS_INSTANTIATE

void set_kernel_events(hipEvent_t start, hipEvent_t stop)
{
    t_start = start;
    t_stop = stop;
    t_used = false;
}

bool take_kernel_events_used()
{
    const bool used = t_used;
    t_start = t_stop = nullptr;
    t_used = false;
    return used;
}

}  // namespace pcs

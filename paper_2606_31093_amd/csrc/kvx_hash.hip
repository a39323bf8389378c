// kvx_hash.hip -- chained page hashes for gfx950 (Omni-Flow Sec. 5.1:
// each page's hash encodes its predecessor's, so equal hashes mean an equal
// prefix page by page).  Definition, with fnv = FNV-1a 64:
//   c_j = fnv(records of page j),   h_j = fnv(le64(h_{j-1}) || le64(c_j)).
//
// One launch on the caller's stream, nothing allocated.  Requests are split
// into groups of up to 64, one group per compute unit at a time, and each
// workgroup has two roles:
//
// - Digest wavefronts (KVX_DIGEST_WAVES of them) hash whole pages, one page
//   per lane: 256 bytes per 64-token page of int32 ids, so this is where
//   the arithmetic is.  They take the group's pages 64 at a time from a
//   counter in LDS, in page-index order across the group's requests (all
//   pages 0, then all pages 1, ...), which is the order the chain needs
//   them in, and write c_j to out[out_off + j].
// - The chain wavefront gives each request of the group one lane.  The lane
//   walks its request's pages in order and overwrites each c_j with h_j:
//   16 bytes hashed per page, strictly in order, so the longest request
//   sets the floor.  It starts as soon as the first digests are written
//   instead of after all of them, which is what one kernel per role would
//   cost.  Its instructions take priority on the SIMD it shares.
//
// The hand-off goes through LDS: each digest wavefront publishes the page
// index of the first page of the chunk it is working on, after a release
// fence for the stores of its previous chunk.  Chunks are handed out in
// order, so every page below the smallest published index has been
// digested in every request of the group.  Digest wavefronts never wait;
// the chain wavefront waits only for them, with a bounded sleep loop that
// raises KVX_DERR_STALLED instead of spinning forever.
//
// out[] holds digests until the chain has passed them: callers see it only
// after the stream has passed the kernel.

#include <stdlib.h>

#include "kvx_hash.h"

namespace kvx {
namespace {

constexpr int kWave = 64;
#ifndef KVX_HASH_BATCH
#define KVX_HASH_BATCH 8    // words in flight per digest lane
#endif
#ifndef KVX_CHAIN_BATCH
#define KVX_CHAIN_BATCH 16  // pages chained per step of the chain lanes
#endif
constexpr uint64_t kBasis = 0xcbf29ce484222325ull;
constexpr uint64_t kPrime = 0x100000001b3ull;

__device__ __forceinline__ uint64_t fnv_word(uint64_t h, uint32_t w) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        h ^= (w >> (8 * b)) & 0xffu;
        h *= kPrime;
    }
    return h;
}

__device__ __forceinline__ uint64_t fnv_u64(uint64_t h, uint64_t v) {
    h = fnv_word(h, (uint32_t)v);
    return fnv_word(h, (uint32_t)(v >> 32));
}

// h_j from h_{j-1} and c_j.
__device__ __forceinline__ uint64_t chain_step(uint64_t h, uint64_t c) {
    return fnv_u64(fnv_u64(kBasis, h), c);
}

// FNV-1a of nw 32-bit words, KVX_HASH_BATCH loads in flight.
__device__ __forceinline__ uint64_t digest(const uint32_t *w, int64_t nw) {
    constexpr int B = KVX_HASH_BATCH;
    uint64_t c = kBasis;
    int64_t i = 0;
    for (; i + B <= nw; i += B) {
        uint32_t v[B];
#pragma unroll
        for (int u = 0; u < B; ++u) v[u] = w[i + u];
#pragma unroll
        for (int u = 0; u < B; ++u) c = fnv_word(c, v[u]);
    }
    for (; i < nw; ++i) c = fnv_word(c, w[i]);
    return c;
}

// A record is used only if its payload range and its out range lie inside
// the caller's buffers; *pages receives its page count.
__device__ __forceinline__ bool valid(const kvx_hash_req &q, const HashParams &p,
                                      int64_t *pages) {
    const int32_t n = q.n_positions;
    *pages = n > 0 ? ((int64_t)n + p.T - 1) / p.T : 0;
    return n >= 0 && q.reserved == 0 && q.payload_off >= 0 &&
           q.payload_off <= p.payload_positions - n && q.out_off >= 0 &&
           q.out_off <= p.out_len - *pages;
}

#ifndef KVX_DIGEST_WAVES
#define KVX_DIGEST_WAVES 7   // digest wavefronts beside the chain wavefront
#endif


constexpr int kDW = KVX_DIGEST_WAVES;
constexpr int kSlots = kWave;              // requests per group at most
constexpr uint64_t kAllDone = ~0ull;

// Shared state of one group of requests.  Items are the pages of the group
// in page-index-major order: all pages 0 of the group's requests, then all
// pages 1 of those that have one, and so on, which is the order in which the
// chain lanes need them.  With the page counts sorted ascending (m[]), the
// requests that have a page j are the ascending positions k..63 for
// m[k-1] <= j < m[k], so item q falls in the segment k with
// base[k] <= q < base[k+1] and each segment is a (page, position) grid.
struct GroupLds {
    int64_t key[kSlots];       // (page count, slot) by slot, for the sort
    int32_t m[kSlots];         // page counts, ascending
    int32_t perm[kSlots];      // ascending position -> slot
    int32_t npos[kSlots];      // n_positions by slot
    int64_t base[kSlots + 1];  // first item of segment k
    int64_t pay[kSlots];       // payload_off by slot
    int64_t outo[kSlots];      // out_off by slot
    uint64_t next;             // first item not yet handed to a digest wavefront
    uint64_t cur[kDW];         // first item of the chunk each digest wavefront is on
};

__global__ void __launch_bounds__(kWave * (1 + kDW)) kvx_page_hash_kernel(HashParams p) {
    __shared__ GroupLds s;
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int64_t wpr = p.rec_bytes / 4;
    const int64_t ngroups = (p.n_reqs + p.group - 1) / p.group;
    for (int64_t g = blockIdx.x; g < ngroups; g += gridDim.x) {
        // The chain wavefront's lane `lane` owns slot `lane` of the group.
        int32_t pages = 0;
        uint64_t seed = 0;
        int pos = 0;
        if (wave == 0) {
            const int64_t r = g * p.group + lane;
            int32_t npos = 0;
            int64_t pay = 0, outo = 0;
            if (lane < p.group && r < p.n_reqs) {
                const kvx_hash_req &q = p.reqs[r];
                int64_t pg;
                if (valid(q, p, &pg)) {
                    pages = (int32_t)pg;
                    seed = q.seed;
                    pay = q.payload_off;
                    outo = q.out_off;
                    npos = q.n_positions;
                } else if (p.err) {
                    atomicOr(p.err, KVX_DERR_BAD_REQ);
                }
            }
            s.key[lane] = ((int64_t)pages << 6) | lane;
            s.npos[lane] = npos;
            s.pay[lane] = pay;
            s.outo[lane] = outo;
        }
        __syncthreads();
        if (wave == 0) {
            // ascending rank of the unique key (pages, slot)
            const int64_t key = ((int64_t)pages << 6) | lane;
#pragma unroll
            for (int t = 0; t < kSlots; ++t) pos += s.key[t] < key;
            s.m[pos] = pages;
            s.perm[pos] = lane;
        }
        __syncthreads();
        if (wave == 0) {
            const int64_t m_prev = lane ? s.m[lane - 1] : 0;
            int64_t v = (s.m[lane] - m_prev) * (int64_t)(kSlots - lane);
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const int64_t t = __shfl_up(v, d);
                if (lane >= d) v += t;
            }
            s.base[lane + 1] = v;
            if (lane == 0) {
                s.base[0] = 0;
                s.next = 0;
            }
            if (lane < kDW) s.cur[lane] = 0;
        }
        __syncthreads();
        const uint64_t total = (uint64_t)s.base[kSlots];
        if (wave > 0) {
            // Digest wavefront: take 64 items at a time, in item order, and
            // publish the page index of the first one.
            const int d = wave - 1;
            for (;;) {
                uint64_t q0 = 0;
                if (lane == 0) q0 = atomicAdd(&s.next, (unsigned long long)kWave);
                q0 = __shfl(q0, 0);
                const uint64_t q = q0 + lane;
                int64_t j = 0;
                int slot = 0;
                if (q < total) {
                    int k = 0;
#pragma unroll
                    for (int step = kSlots / 2; step > 0; step >>= 1)
                        if ((uint64_t)s.base[k + step] <= q) k += step;
                    const uint64_t off = q - (uint64_t)s.base[k];
                    const uint32_t act = kSlots - k;
                    uint64_t jo, ro;
                    if (off < (1ull << 32)) {
                        jo = (uint32_t)off / act;
                        ro = (uint32_t)off - (uint32_t)jo * act;
                    } else {
                        jo = off / act;
                        ro = off - jo * act;
                    }
                    j = (k ? s.m[k - 1] : 0) + (int64_t)jo;
                    slot = s.perm[k + (int)ro];
                }
                const int64_t row = __shfl(j, 0);
                // the digests of the previous chunk are in memory before the
                // chain wavefront can see that this wavefront has moved on
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                if (lane == 0)
                    __hip_atomic_store(&s.cur[d], q0 < total ? (uint64_t)row : kAllDone,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                if (q0 >= total) break;
                if (q < total) {
                    const int64_t first = j * p.T;
                    const int64_t n = s.npos[slot];
                    const int64_t count = n - first < p.T ? n - first : p.T;
                    p.out[s.outo[slot] + j] =
                        digest(p.payload + (s.pay[slot] + first) * wpr, count * wpr);
                }
            }
        } else {
            // Chain wavefront: lane `lane` walks its request's pages in order,
            // up to KVX_CHAIN_BATCH at a time, as their digests arrive.
            // While one batch is chained the next one's digests are loaded if
            // they are already written.  Its instructions go first on the
            // SIMD it shares with digest wavefronts: the chain is the critical
            // path, the digests fill the gaps.
            constexpr int B = KVX_CHAIN_BATCH;
            __builtin_amdgcn_s_setprio(3);
            // Loads are issued for every lane, with indices clamped into the
            // lane's own pages (page 0 of out for a lane without pages, which
            // exists whenever any lane has pages), so the compiler can count
            // the loads in flight and wait only for the batch it needs.
            const bool act = pages > 0;
            const uint64_t *src = act ? p.out + s.outo[lane] : p.out;
            uint64_t *o = p.out + s.outo[lane];
            const int64_t last = act ? pages - 1 : 0;
            uint64_t h = seed;
            int64_t j = 0;
            int pf = 0;                     // digests of pages [j, j + pf) are in cn[]
            uint64_t cn[B];
#pragma unroll
            for (int u = 0; u < B; ++u) cn[u] = 0;
            uint64_t idle = 0;
            const uint64_t idle_limit = p.idle_limit;
            while (__any(j < pages)) {
                uint64_t lim = kAllDone;
#pragma unroll
                for (int d = 0; d < kDW; ++d) {
                    const uint64_t c = __hip_atomic_load(&s.cur[d], __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_WORKGROUP);
                    lim = c < lim ? c : lim;
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
                // pages [j, ready) are digested
                const int64_t ready = (uint64_t)pages < lim ? (int64_t)pages : (int64_t)lim;
                int take = pf;
                if (pf == 0 && j < ready) take = ready - j < B ? (int)(ready - j) : B;
                if (!__any(take > 0)) {
                    if (++idle > idle_limit) {
                        if (lane == 0 && p.err) atomicOr(p.err, KVX_DERR_STALLED);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                    continue;
                }
                idle = 0;
                uint64_t c[B];
                if (__any(pf == 0 && take > 0)) {
#pragma unroll
                    for (int u = 0; u < B; ++u) {
                        const int64_t i = j + u < last ? j + u : last;
                        c[u] = src[i];
                    }
#pragma unroll
                    for (int u = 0; u < B; ++u) c[u] = pf ? cn[u] : c[u];
                } else {
#pragma unroll
                    for (int u = 0; u < B; ++u) c[u] = cn[u];
                }
                // the digests after this batch that are already written
                const int64_t j2 = j + take;
                pf = j2 < ready ? (ready - j2 < B ? (int)(ready - j2) : B) : 0;
#pragma unroll
                for (int u = 0; u < B; ++u) {
                    const int64_t i = j2 + u < last ? j2 + u : last;
                    cn[u] = src[i];
                }
#pragma unroll
                for (int u = 0; u < B; ++u) {
                    if (u < take) {
                        h = chain_step(h, c[u]);
                        o[j + u] = h;
                    }
                }
                j = j2;
            }
            __builtin_amdgcn_s_setprio(0);
        }
        __syncthreads();   // the next group reuses the shared state
    }
}

}  // namespace

int launch_hash(const HashParams &p0, hipStream_t stream) {
    if (p0.n_reqs == 0) return hipSuccess;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    HashParams p = p0;
    // Empty polls in a row the chain allows: far more than one page's digest
    // takes, even with the payload in host memory.  A build with
    // KVX_HASH_IDLE_POLLS defined uses that bound instead (a test library
    // built with a bound of 1 sees the chain give up cleanly).
#ifdef KVX_HASH_IDLE_POLLS
    p.idle_limit = (uint64_t)(KVX_HASH_IDLE_POLLS);
#else
    p.idle_limit = (1ull << 22) + 64ull * (uint64_t)p.T * (uint64_t)p.rec_bytes;
#endif
    // one group per compute unit, each of at most 64 requests
    const int32_t group = (p.n_reqs + cus - 1) / cus;
    p.group = group < 1 ? 1 : group > kSlots ? kSlots : group;
    const int64_t ngroups = (p.n_reqs + p.group - 1) / p.group;
    const int grid = ngroups < cus ? (int)ngroups : cus;
    hipLaunchKernelGGL(kvx_page_hash_kernel, dim3(grid), dim3(kWave * (1 + kDW)), 0, stream, p);
    return hipGetLastError();
}

}  // namespace kvx

// kvx_hash.hip -- chained page hashes for gfx950 (Omni-Flow Sec. 5.1:
// each page's hash encodes its predecessor's, so equal hashes mean an equal
// prefix page by page).  Definition, with fnv = FNV-1a 64:
//   c_j = fnv(records of page j),   h_j = fnv(le64(h_{j-1}) || le64(c_j)).
//
// Two launches on the caller's stream, nothing allocated:
//
// 1. Digests.  One wavefront per request (a grid-stride loop over
//    requests); pages are taken 64 at a time and lane j computes c_j,
//    issuing its page's loads KVX_HASH_BATCH words at a time before hashing
//    them.  Larger batches fetch the lines that neighbouring pages share
//    fewer times but hold more registers, so fewer wavefronts hide load
//    latency; 32 words (128 bytes) is the measured balance.  c_j goes to
//    out[out_off + j], 64 pages per coalesced store.  This is where the
//    arithmetic is: 256 bytes hashed per 64-token page of int32 ids.
//
// 2. Chain.  One lane per request: the lane walks its request's digests in
//    page order and overwrites each with h_j.  16 bytes hashed per page, but
//    strictly in order.  With a lane per request the chain costs one vector
//    instruction stream per 64 requests; run inside the digest wavefronts it
//    would be one scalar instruction stream per request, and the scalar unit
//    a compute unit's wavefronts share becomes the bottleneck.
//
// Between the two launches out[] holds the digests: callers see it only
// after the stream has passed both.

#include "kvx_hash.h"

namespace kvx {
namespace {

constexpr int kWave = 64;
#ifndef KVX_HASH_BATCH
#define KVX_HASH_BATCH 32   // words in flight per lane in the digest
#endif
#ifndef KVX_CHAIN_BATCH
#define KVX_CHAIN_BATCH 16  // digests in flight per lane in the chain
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

__global__ void __launch_bounds__(kWave) kvx_page_digest_kernel(HashParams p) {
    const int lane = threadIdx.x;
    const int64_t wpr = p.rec_bytes / 4;
    for (int32_t r = blockIdx.x; r < p.n_reqs; r += gridDim.x) {
        const kvx_hash_req &q = p.reqs[r];
        int64_t pages;
        if (!valid(q, p, &pages)) {
            if (lane == 0 && p.err) atomicOr(p.err, KVX_DERR_BAD_REQ);
            continue;                       // uniform across the wavefront
        }
        const int32_t n = q.n_positions;
        for (int64_t j = lane; j < pages; j += kWave) {
            const int64_t first = j * p.T;
            const int64_t count = n - first < p.T ? n - first : p.T;
            p.out[q.out_off + j] = digest(p.payload + (q.payload_off + first) * wpr, count * wpr);
        }
    }
}

__global__ void __launch_bounds__(kWave) kvx_page_chain_kernel(HashParams p) {
    constexpr int B = KVX_CHAIN_BATCH;
    for (int64_t r = (int64_t)blockIdx.x * kWave + threadIdx.x; r < p.n_reqs;
         r += (int64_t)gridDim.x * kWave) {
        const kvx_hash_req &q = p.reqs[r];
        int64_t pages;
        if (!valid(q, p, &pages)) continue;     // flagged by the digest launch
        uint64_t *o = p.out + q.out_off;
        uint64_t h = q.seed;
        uint64_t next[B];
#pragma unroll
        for (int u = 0; u < B; ++u) next[u] = u < pages ? o[u] : 0;
        for (int64_t j = 0; j < pages; j += B) {
            uint64_t c[B];
#pragma unroll
            for (int u = 0; u < B; ++u) c[u] = next[u];
            // the following batch is in flight while this one is chained
#pragma unroll
            for (int u = 0; u < B; ++u) next[u] = j + B + u < pages ? o[j + B + u] : 0;
#pragma unroll
            for (int u = 0; u < B; ++u) {
                if (j + u < pages) {
                    h = chain_step(h, c[u]);
                    o[j + u] = h;
                }
            }
        }
    }
}

}  // namespace

int launch_hash(const HashParams &p, hipStream_t stream) {
    if (p.n_reqs == 0) return hipSuccess;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int digest_grid = p.n_reqs < cus * 32 ? p.n_reqs : cus * 32;
    hipLaunchKernelGGL(kvx_page_digest_kernel, dim3(digest_grid), dim3(kWave), 0, stream, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int chain_blocks = (p.n_reqs + kWave - 1) / kWave;
    const int chain_grid = chain_blocks < cus * 8 ? chain_blocks : cus * 8;
    hipLaunchKernelGGL(kvx_page_chain_kernel, dim3(chain_grid), dim3(kWave), 0, stream, p);
    return hipGetLastError();
}

}  // namespace kvx

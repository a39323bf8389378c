// kvx_hash.h -- launch parameters of the chained page hash kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvx.h"

namespace kvx {

struct HashParams {
    const uint32_t *payload;      // records as 32-bit words
    int64_t payload_positions;    // records in the payload
    int32_t rec_bytes;            // a multiple of 4
    int32_t T;                    // positions per page
    const kvx_hash_req *reqs;
    int32_t n_reqs;
    uint64_t *out;
    int64_t out_len;
    uint32_t *err;
    int32_t group;                // requests per workgroup
    uint64_t idle_limit;          // empty polls in a row before the chain gives up
};

int launch_hash(const HashParams &p, hipStream_t stream);

}  // namespace kvx

// Device-coherent 16-byte accesses for data exchanged between persistent
// workgroups (possibly on different XCDs, whose L2 caches are not coherent
// with each other).  Cache policy SC1 is the one agent-scope atomics use:
// stores write through to the device coherence point and loads read from
// it.  A producer that stores its shared data this way, waits for the
// stores to complete (s_waitcnt vmcnt(0)) and then raises a flag with an
// agent-scope atomic needs no L2 writeback, and a consumer that sees the
// flag and loads the shared data this way needs no L2 invalidate; all other
// data stays cached.  Addresses are float indices into a raw buffer
// resource whose byte size fits 31 bits.
#pragma once

#include <hip/hip_runtime.h>

namespace plstm {

typedef float cf4 __attribute__((ext_vector_type(4)));

constexpr int kBufferRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data
constexpr int kCachePolicySC1 = 16;

__device__ inline __amdgpu_buffer_rsrc_t coherent_rsrc(const float *base, long long nfloats)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), (short)0,
                                             (int)(nfloats * (long long)sizeof(float)),
                                             kBufferRsrcWord3);
}

__device__ inline cf4 load_coherent(__amdgpu_buffer_rsrc_t rs, int idx)
{
    return __builtin_bit_cast(
        cf4, __builtin_amdgcn_raw_buffer_load_b128(rs, idx * (int)sizeof(float), 0,
                                                    kCachePolicySC1));
}

__device__ inline void store_coherent(__amdgpu_buffer_rsrc_t rs, int idx, cf4 v)
{
    typedef unsigned u4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), rs,
                                           idx * (int)sizeof(float), 0, kCachePolicySC1);
}

}  // namespace plstm

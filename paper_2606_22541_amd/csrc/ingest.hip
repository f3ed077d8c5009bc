// Asynchronous ingest (section 3.2.1): the senders of a micro-batch write
// their token rows into statically allocated receive buffers and then raise
// a ready word each (the per-sender bits of the bitmap in Table 2).  The MoE
// side enqueues its work ahead of time behind a device-side wait on those
// words, so the stage starts as soon as the rows are complete, without a
// host round trip.
//
// The wait is a one-wave kernel that polls the words with agent-scope
// acquire loads and sleeps between polls.  It is bounded: after spin_limit
// polls it sets an error bit and exits, so every launch terminates whether
// or not the senders ever signal.  A ready word counts rounds (epochs): the
// wait holds until every word has reached the round's epoch, compared as a
// wrapping 32-bit counter, so words never need clearing between rounds.
#include "kernels.h"

namespace moe {

namespace {

__device__ __forceinline__ bool reached(uint32_t v, uint32_t epoch)
{
    return (int32_t)(v - epoch) >= 0;
}

__global__ __launch_bounds__(64)
void k_ingest_wait(const uint32_t *__restrict__ ready, int32_t n_words, uint32_t epoch,
                   uint32_t spin_limit, int32_t *__restrict__ err)
{
    const int lane = threadIdx.x;
    for (uint32_t spins = 0;; ++spins) {
        bool ok = true;
        for (int i = lane; i < n_words; i += 64)
            ok = ok && reached(__hip_atomic_load(ready + i, __ATOMIC_ACQUIRE,
                                                 __HIP_MEMORY_SCOPE_AGENT),
                               epoch);
        if (__all(ok)) break;
        if (spins + 1 >= spin_limit) {
            if (lane == 0) atomicOr(err, kErrIngestTimeout);
            break;
        }
        __builtin_amdgcn_s_sleep(16);
    }
}

__global__ __launch_bounds__(64)
void k_ingest_signal(uint32_t *__restrict__ word, uint32_t epoch)
{
    // earlier work on the stream has completed and been released at its
    // kernel boundaries; the release store orders this kernel's view as well
    if (threadIdx.x == 0)
        __hip_atomic_store(word, epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

hipError_t launch_ingest_wait(const uint32_t *ready, int32_t n_words, uint32_t epoch,
                              uint32_t spin_limit, int32_t *err, hipStream_t s)
{
    hipLaunchKernelGGL(k_ingest_wait, dim3(1), dim3(64), 0, s, ready, n_words, epoch,
                       spin_limit, err);
    return hipGetLastError();
}

hipError_t launch_ingest_signal(uint32_t *word, uint32_t epoch, hipStream_t s)
{
    hipLaunchKernelGGL(k_ingest_signal, dim3(1), dim3(64), 0, s, word, epoch);
    return hipGetLastError();
}

}  // namespace moe

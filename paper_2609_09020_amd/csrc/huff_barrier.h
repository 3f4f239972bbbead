// One-shot hand-off between the workgroups of a single launch, for the
// entropy decoder's one-launch path: every workgroup arrives once; the last
// to arrive runs a serial step (the repair of subsequences a workgroup could
// not settle) and then releases the others, which wait for it a bounded time.
//
// State: one 64-bit word, generation << 32 | flagged << 16 | arrivals, zero
// when the handle is created.  A workgroup arrives with one atomic add, which
// also returns the generation it arrived in; a workgroup that has something
// for the serial step adds one to `flagged` in the same add.  The last
// arrival (arrivals == n - 1) owns the serial step and learns from the value
// it read whether any workgroup flagged one; when done it stores
// (generation + 1) << 32: count and flags are back at zero for the next
// launch, and the waiters, spinning on the generation, go on.  Nothing is
// cleared between launches (a replayed launch finds the word as the previous
// one left it), and a waiter that gives up leaves the word consistent: the
// last arrival still resets it.  At most 65535 workgroups arrive.
//
// The last arrival can only come once every workgroup has started: a waiter
// that holds a CU while others of the launch wait for one could wait for
// ever, so a waiter stops after a time limit and reports it.
//
// Leaving: a second word, error bits << 32 | departures, also zero at
// create.  Every workgroup leaves once, after its last write, whatever path
// it took (a waiter that gave up included): it ors its error bits into the
// word, then counts itself; the last to leave receives every workgroup's
// bits and resets the word.  Error bits of a waiter that gives up go this
// way, not straight into the caller's status, which the launch's first
// workgroup may clear later than the waiter gives up.
//
// The protocol is written once over an operations policy, so that the host
// can run it with std::atomic and threads (its tests) and the kernel with
// device-scope atomics:
//   uint64_t Ops::fetch_add(uint64_t *w, uint64_t v)   returns the old value
//   void     Ops::fetch_or(uint64_t *w, uint64_t v)
//   uint64_t Ops::load(const uint64_t *w)
//   void     Ops::store(uint64_t *w, uint64_t v)
//   void     Ops::pause()                               between polls
//   uint64_t Ops::now()                                 a clock the wait's limit is in
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define PIC_HD __host__ __device__
#else
#define PIC_HD
#endif

namespace pic {
namespace huff_barrier {

struct Arrival {
    uint32_t generation;   // the generation the caller arrived in
    bool last;             // the caller arrived last: it owns the serial step
    bool flagged;          // (last only) some workgroup, the caller included, flagged
};

// Arrive; one call per workgroup and launch.  `n` is the number of
// workgroups of the launch (1 .. 65535); `flag`: the caller has something
// for the serial step.
template <class Ops>
PIC_HD inline Arrival arrive(uint64_t *word, uint32_t n, bool flag)
{
    const uint64_t old = Ops::fetch_add(word, flag ? 0x10001u : 1u);
    Arrival a;
    a.generation = (uint32_t)(old >> 32);
    a.last = (old & 0xffffu) == n - 1u;
    a.flagged = flag || ((old >> 16) & 0xffffu) != 0;
    return a;
}

// The last arrival, after its serial step: open the next generation.
template <class Ops>
PIC_HD inline void release(uint64_t *word, const Arrival &a)
{
    Ops::store(word, (uint64_t)(a.generation + 1u) << 32);
}

// A waiter: poll until the generation it arrived in has ended, for at most
// `limit` units of Ops::now().  True when released, false when it gave up.
template <class Ops>
PIC_HD inline bool wait(const uint64_t *word, const Arrival &a, uint64_t limit)
{
    const uint64_t t0 = Ops::now();
    while (Ops::now() - t0 < limit) {
        if ((uint32_t)(Ops::load(word) >> 32) != a.generation)
            return true;
        Ops::pause();
    }
    return (uint32_t)(Ops::load(word) >> 32) != a.generation;
}

// Leave; one call per workgroup and launch, after its last write.  True for
// the last to leave, which receives in *all_err the error bits every
// workgroup left with (the word is then reset for the next launch).
template <class Ops>
PIC_HD inline bool leave(uint64_t *word, uint32_t n, uint32_t err, uint32_t *all_err)
{
    if (err)
        Ops::fetch_or(word, (uint64_t)err << 32);
    const uint64_t old = Ops::fetch_add(word, 1u);   // after the or: one location, one order
    if ((uint32_t)old != n - 1u)
        return false;
    *all_err = (uint32_t)(old >> 32);
    Ops::store(word, 0);
    return true;
}

#if defined(__HIPCC__)
// The kernels' policy: device-scope atomics on the scratch words (one
// coherent place for every XCD), a short sleep between polls, the wait's
// limit in ticks of the 100 MHz real-time counter.
struct DeviceOps {
    __device__ static uint64_t fetch_add(uint64_t *w, uint64_t v)
    {
        return __hip_atomic_fetch_add(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ static void fetch_or(uint64_t *w, uint64_t v)
    {
        (void)__hip_atomic_fetch_or(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ static uint64_t load(const uint64_t *w)
    {
        return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ static void store(uint64_t *w, uint64_t v)
    {
        __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ static void pause() { __builtin_amdgcn_s_sleep(2); }
    __device__ static uint64_t now() { return __builtin_amdgcn_s_memrealtime(); }
};
#endif

}  // namespace huff_barrier
}  // namespace pic

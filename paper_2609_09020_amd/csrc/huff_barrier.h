// One-shot hand-off between the workgroups of a single launch, for the
// entropy decoder's one-launch path: every workgroup arrives once; the last
// to arrive runs a serial step (the repair of subsequences a workgroup could
// not settle) and then releases the others, which wait for it a bounded time.
//
// State: one 64-bit word, generation << 32 | arrivals, zero when the handle
// is created.  A workgroup arrives with one atomic add, which also returns
// the generation it arrived in.  The last arrival (arrivals == n - 1) owns
// the serial step; when done it stores (generation + 1) << 32: the count is
// back at zero for the next launch, and the waiters, spinning on the
// generation, go on.  Nothing is cleared between launches (a replayed launch
// finds the word as the previous one left it), and a waiter that gives up
// leaves the word consistent: the last arrival still resets it.
//
// The last arrival can only come once every workgroup has started: a waiter
// that holds a CU while others of the launch wait for one could wait for
// ever, so a waiter stops after `spin_limit` polls and reports it.
//
// The protocol is written once over an operations policy, so that the host
// can run it with std::atomic and threads (its tests) and the kernel with
// device-scope atomics:
//   uint64_t Ops::fetch_add(uint64_t *w, uint64_t v)   returns the old value
//   uint64_t Ops::load(const uint64_t *w)
//   void     Ops::store(uint64_t *w, uint64_t v)
//   void     Ops::pause()                               between polls
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
};

// Arrive; one call per workgroup and launch.  `n` is the number of
// workgroups of the launch (>= 1).
template <class Ops>
PIC_HD inline Arrival arrive(uint64_t *word, uint32_t n)
{
    const uint64_t old = Ops::fetch_add(word, 1u);
    Arrival a;
    a.generation = (uint32_t)(old >> 32);
    a.last = (uint32_t)old == n - 1u;
    return a;
}

// The last arrival, after its serial step: open the next generation.
template <class Ops>
PIC_HD inline void release(uint64_t *word, const Arrival &a)
{
    Ops::store(word, (uint64_t)(a.generation + 1u) << 32);
}

// A waiter: poll until the generation it arrived in has ended, at most
// `spin_limit` times.  True when released, false when it gave up.
template <class Ops>
PIC_HD inline bool wait(const uint64_t *word, const Arrival &a, uint32_t spin_limit)
{
    for (uint32_t i = 0; i < spin_limit; ++i) {
        if ((uint32_t)(Ops::load(word) >> 32) != a.generation)
            return true;
        Ops::pause();
    }
    return (uint32_t)(Ops::load(word) >> 32) != a.generation;
}

}  // namespace huff_barrier
}  // namespace pic

// Host run of the entropy decoder's one-launch hand-off protocol
// (paper_2609_09020_amd/csrc/huff_barrier.h), with threads as workgroups and
// GCC atomics as the operations policy.  Prints one line per scenario;
// exits non-zero on the first failed check.
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include "huff_barrier.h"

namespace hb = pic::huff_barrier;

static thread_local unsigned long long polls = 0;

struct HostOps {
    static uint64_t fetch_add(uint64_t *w, uint64_t v) { return __atomic_fetch_add(w, v, __ATOMIC_SEQ_CST); }
    static void fetch_or(uint64_t *w, uint64_t v) { (void)__atomic_fetch_or(w, v, __ATOMIC_SEQ_CST); }
    static uint64_t load(const uint64_t *w) { return __atomic_load_n(w, __ATOMIC_SEQ_CST); }
    static void store(uint64_t *w, uint64_t v) { __atomic_store_n(w, v, __ATOMIC_SEQ_CST); }
    static void pause()
    {
        ++polls;
        std::this_thread::yield();
    }
    // the wait's limit counted in polls here
    static uint64_t now() { return polls; }
};

#define CHECK(c, ...)                                                   \
    do {                                                                \
        if (!(c)) {                                                     \
            std::printf("FAIL line %d: ", __LINE__);                     \
            std::printf(__VA_ARGS__);                                   \
            std::printf("\n");                                          \
            std::exit(1);                                               \
        }                                                               \
    } while (0)

// One launch of n workgroups.  The last arrival writes `payload` (its serial
// step) after `delay_ms`, then releases unless `no_release`.  Returns how
// many waiters were released and how many gave up; `max_polls` receives the
// largest poll count of a waiter.
struct Outcome {
    int released = 0, gave_up = 0, saw_payload = 0, lasts = 0;
    bool last_flagged = false;
    unsigned long long max_polls = 0;
};

// flags: bit i set when workgroup i (< 64) flags something for the serial step
static Outcome launch(uint64_t *word, int n, uint32_t spin_limit, int delay_ms, bool no_release,
                      int *payload, int value, uint64_t flags = 0)
{
    Outcome o;
    std::atomic<int> released{0}, gave_up{0}, saw{0}, lasts{0};
    std::atomic<bool> last_flagged{false};
    std::atomic<unsigned long long> maxp{0};
    std::vector<std::thread> ts;
    for (int i = 0; i < n; ++i)
        ts.emplace_back([&, i] {
            polls = 0;
            const hb::Arrival a = hb::arrive<HostOps>(word, (uint32_t)n, i < 64 && ((flags >> i) & 1u));
            if (a.last) {
                ++lasts;
                last_flagged = a.flagged;
                if (delay_ms)
                    std::this_thread::sleep_for(std::chrono::milliseconds(delay_ms));
                __atomic_store_n(payload, value, __ATOMIC_SEQ_CST);
                if (!no_release)
                    hb::release<HostOps>(word, a);
                return;
            }
            if (hb::wait<HostOps>(word, a, spin_limit)) {
                ++released;
                if (__atomic_load_n(payload, __ATOMIC_SEQ_CST) == value)
                    ++saw;
            } else {
                ++gave_up;
            }
            unsigned long long p = polls, cur = maxp.load();
            while (p > cur && !maxp.compare_exchange_weak(cur, p)) {
            }
        });
    for (auto &t : ts)
        t.join();
    o.released = released;
    o.gave_up = gave_up;
    o.saw_payload = saw;
    o.lasts = lasts;
    o.last_flagged = last_flagged;
    o.max_polls = maxp;
    return o;
}

int main()
{
    uint64_t word = 0;   // as the handle's scratch starts
    int payload = 0;

    // 1. every waiter is released and sees the serial step's result; the
    //    word then holds generation 1, count 0
    {
        const Outcome o = launch(&word, 16, 1u << 30, 5, false, &payload, 1);
        CHECK(o.lasts == 1, "one last arrival, got %d", o.lasts);
        CHECK(o.released == 15 && o.gave_up == 0, "released %d gave up %d", o.released, o.gave_up);
        CHECK(o.saw_payload == 15, "saw the serial step's result: %d", o.saw_payload);
        CHECK(word == (1ull << 32), "word %llx", (unsigned long long)word);
        std::printf("release: 16 workgroups, 15 released, word %llx\n", (unsigned long long)word);
    }
    // 2. launches in a row, with different workgroup counts, no clearing
    //    between them (a replayed launch)
    for (int g = 0; g < 200; ++g) {
        const int n = 1 + g % 64;
        const Outcome o = launch(&word, n, 1u << 30, 0, false, &payload, 100 + g);
        CHECK(o.lasts == 1 && o.released == n - 1 && o.saw_payload == n - 1, "launch %d", g);
    }
    CHECK(word == (201ull << 32), "word after 201 launches %llx", (unsigned long long)word);
    std::printf("replay: 200 more launches of 1..64 workgroups, word %llx\n", (unsigned long long)word);

    // 3. a spin limit of 0: every waiter gives up at once (the condition a
    //    caller can force), the last arrival still resets the word, and the
    //    next launch works
    {
        const Outcome o = launch(&word, 16, 0, 20, false, &payload, 7);
        CHECK(o.gave_up + o.released == 15, "every waiter returned");
        CHECK(o.max_polls == 0, "no poll with a limit of 0: %llu", o.max_polls);
        CHECK(word == (202ull << 32), "word consistent after give-ups %llx", (unsigned long long)word);
        const Outcome o2 = launch(&word, 16, 1u << 30, 0, false, &payload, 8);
        CHECK(o2.released == 15, "next launch released %d", o2.released);
        std::printf("forced give-up: %d of 15 gave up, word consistent, next launch released 15\n", o.gave_up);
    }
    // 4. the bound: the last arrival never releases; every waiter returns
    //    after exactly spin_limit polls
    {
        const uint32_t lim = 1000;
        const Outcome o = launch(&word, 8, lim, 0, true, &payload, 9);
        CHECK(o.gave_up == 7 && o.released == 0, "gave up %d released %d", o.gave_up, o.released);
        CHECK(o.max_polls == lim, "polls %llu", o.max_polls);
        std::printf("bound: 7 waiters gave up after %llu polls each (limit %u)\n", o.max_polls, lim);
    }
    // 5. flags: the last arrival learns whether any workgroup (itself
    //    included, whichever arrives last) flagged the serial step, and the
    //    release clears the flags with the count
    {
        uint64_t fword = 0, gen = 0;   // (the bound above left its word unreleased on purpose)
        const uint64_t patterns[] = {0ull, 1ull, 1ull << 63, 0x5555555555555555ull, ~0ull, 1ull << 17};
        for (int g = 0; g < 120; ++g) {
            const int n = 1 + g % 64;
            const uint64_t f = patterns[g % 6] & (n == 64 ? ~0ull : ((1ull << n) - 1));
            const Outcome o = launch(&fword, n, 1u << 30, 0, false, &payload, 300 + g, f);
            CHECK(o.lasts == 1 && o.released == n - 1, "flag launch %d", g);
            CHECK(o.last_flagged == (f != 0), "launch %d: flagged %d, want %d", g, (int)o.last_flagged, (int)(f != 0));
            ++gen;
            CHECK(fword == gen << 32, "launch %d: word %llx", g, (unsigned long long)fword);
        }
        std::printf("flags: 120 launches of 1..64 workgroups, the last arrival saw every flag, word reset\n");
    }
    // 6. leaving: every workgroup once, some with error bits; exactly one
    //    last, which gets every bit, and the word is zero again; repeated
    {
        uint64_t leave_word = 0;
        for (int g = 0; g < 100; ++g) {
            const int n = 1 + g % 64;
            std::atomic<int> lasts{0};
            std::atomic<uint32_t> got{0};
            uint32_t want = 0;
            std::vector<std::thread> ts;
            for (int i = 0; i < n; ++i) {
                const uint32_t err = (i % 7 == 3) ? (1u << (i % 4)) : 0u;
                want |= err;
                ts.emplace_back([&, err] {
                    uint32_t all = 0;
                    if (hb::leave<HostOps>(&leave_word, (uint32_t)n, err, &all)) {
                        ++lasts;
                        got = all;
                    }
                });
            }
            for (auto &t : ts)
                t.join();
            CHECK(lasts == 1, "launch %d: %d last leavers", g, lasts.load());
            CHECK(got == want, "launch %d: bits %x, want %x", g, got.load(), want);
            CHECK(leave_word == 0, "launch %d: word %llx", g, (unsigned long long)leave_word);
        }
        std::printf("leave: 100 launches of 1..64 workgroups, one last leaver each with every error bit\n");
    }
    std::printf("OK\n");
    return 0;
}

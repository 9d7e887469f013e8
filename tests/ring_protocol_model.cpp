// Host model of the warp-specialised kernel's circular-buffer protocol (test
// infrastructure; built with g++ and run under ThreadSanitizer by
// tests/test_ring_protocol.py).
//
// NP producer threads and NC consumer threads stand for the producer and
// consumer waves of one workgroup.  They walk T K-iterations through a ring
// of P slots with the slot / counter arithmetic the kernels use
// (paper_2506_11209_amd/csrc/ws_ring.hpp): a producer of K-iteration q waits
// until empty[slot] reaches ring_empty_target, writes its share of the slot
// (plain, non-atomic stores), then signals full[slot] with a release add; a
// consumer waits until full[slot] reaches ring_full_target (acquire), reads
// every share and checks its tags, then releases with an add on empty[slot].
// Half of the consumers walk the ring with the closed forms, half with
// ring_advance, as the two consumer variants of the kernel do.
//
// Waits are bounded (a watchdog like the kernel's, here in milliseconds of
// waiting): on timeout the thread raises an abort flag and every thread
// leaves at its next poll.
//
// Exit status: 0 all tags read as written; 1 a tag mismatch; 2 a wait timed
// out; 3 bad arguments.  ThreadSanitizer reports races on the slot data
// (and exits with its own status) when the ordering is wrong.
//
// With a sixth argument LAG the model follows the LDS-DMA producer and the
// kernels' consumers more closely: a producer signals K-iteration q only
// once it has written q + LAG (its loads stay in flight until then), and
// before it blocks on the slot of q - P (to write q) it signals every
// pending K-iteration, as the kernel does; a consumer checks that
// K-iteration q + 1 is full before it releases q.  The least a blocked
// producer may signal is every pending K-iteration up to q - P + 1 (the
// consumers need it to release q - P); PLANT_SHORT_DRAIN stops one short of
// that.
//
// Planted mistakes, selected with -D for the tests that must catch them:
//   PLANT_EARLY_RELEASE  consumers release the slot before reading it
//   PLANT_EARLY_READ     consumers wait for one producer signal too few
//   PLANT_DROP_SIGNAL    producer 0 skips its signal of K-iteration T/2
//   PLANT_SHORT_DRAIN    (with LAG) a blocked producer signals pending
//                        K-iterations only up to q - P
//   PLANT_PEEK_WRONG_SLOT the counter read with a signal is the signalled
//                        slot's, not the next one's
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include "ws_ring.hpp"

namespace {

constexpr int kChunks = 8;  // words each producer writes per slot use

struct Ring {
  uint32_t P, NP, NC, T;
  int lag = -1;  // < 0: signal each K-iteration as soon as it is written
  long long limit_ms;
  std::vector<std::atomic<uint32_t>> full, empty;
  std::vector<uint64_t> data;  // [P][NP][kChunks], plain memory
  std::atomic<int> abort{0};
  std::atomic<int> timeouts{0}, mismatches{0};
  Ring(uint32_t p, uint32_t np, uint32_t nc, uint32_t t, long long limit)
      : P(p), NP(np), NC(nc), T(t), limit_ms(limit), full(p), empty(p),
        data((size_t)p * np * kChunks, 0) {
    for (auto& c : full) c.store(0);
    for (auto& c : empty) c.store(0);
  }
  uint64_t* share(uint32_t slot, uint32_t producer) {
    return &data[((size_t)slot * NP + producer) * kChunks];
  }
};

uint64_t tag(uint32_t q, uint32_t producer, int chunk) {
  return ((uint64_t)q << 20) ^ ((uint64_t)producer << 8) ^ (uint64_t)chunk ^ 0x5a5a000000000000ull;
}

// true when ctr reached target; false after the watchdog (or another
// thread's) abort.
bool wait_for(Ring& r, std::atomic<uint32_t>& ctr, uint32_t target) {
  const auto start = std::chrono::steady_clock::now();
  long long spins = 0;
  while ((int32_t)(ctr.load(std::memory_order_acquire) - target) < 0) {
    if (r.abort.load(std::memory_order_relaxed)) return false;
    if ((++spins & 255) == 0) {
      const auto waited = std::chrono::steady_clock::now() - start;
      if (std::chrono::duration_cast<std::chrono::milliseconds>(waited).count() > r.limit_ms) {
        r.timeouts.fetch_add(1);
        r.abort.store(1);
        return false;
      }
      std::this_thread::yield();
    }
  }
  return true;
}

// The register-staged producer: it walks the slots incrementally and, with
// each signal, reads the empty[] counter of the slot it writes next; it
// waits on that slot only when the value read does not already reach the
// target (the counters are monotonic).
void producer(Ring& r, uint32_t p) {
  uint32_t w_slot = 0, w_need = 0, seen = 0;
  for (uint32_t q = 0; q < r.T; ++q) {
    const uint32_t slot = w_slot;
    if (slot != wsg::ring_slot(q, r.P) || w_need != wsg::ring_empty_target(q, r.P, r.NC)) {
      r.mismatches.fetch_add(1);  // the incremental walk disagrees with the closed forms
      return;
    }
    if ((int32_t)(seen - w_need) < 0 && !wait_for(r, r.empty[slot], w_need)) return;
    uint64_t* d = r.share(slot, p);
    for (int c = 0; c < kChunks; ++c) d[c] = tag(q, p, c);
    if (++w_slot == r.P) {
      w_slot = 0;
      w_need += r.NC;
    }
#ifdef PLANT_DROP_SIGNAL
    if (!(p == 0 && q == r.T / 2))  // only the signal goes missing; the peek below still runs
#endif
      r.full[slot].fetch_add(1, std::memory_order_release);
#ifdef PLANT_PEEK_WRONG_SLOT
    seen = r.empty[slot].load(std::memory_order_acquire);
#else
    seen = r.empty[w_slot].load(std::memory_order_acquire);
#endif
  }
}

// Producer with deferred signals (LAG >= 0); the drain before a blocking
// wait keeps the consumers' one-K-iteration look-ahead satisfied.
void producer_deferred(Ring& r, uint32_t p) {
  const uint32_t lag = (uint32_t)r.lag;
  uint32_t q_sig = 0;
  auto publish = [&]() {
    r.full[wsg::ring_slot(q_sig, r.P)].fetch_add(1, std::memory_order_release);
    ++q_sig;
  };
  for (uint32_t q = 0; q < r.T; ++q) {
    const uint32_t slot = wsg::ring_slot(q, r.P);
    if (wsg::ring_use(q, r.P) > 0) {
      const uint32_t need = wsg::ring_empty_target(q, r.P, r.NC);
      if ((int32_t)(r.empty[slot].load(std::memory_order_acquire) - need) < 0) {
#ifdef PLANT_SHORT_DRAIN
        while (q_sig + r.P <= q) publish();
#else
        while (q_sig < q) publish();
#endif
        if (!wait_for(r, r.empty[slot], need)) return;
      }
    }
    uint64_t* d = r.share(slot, p);
    for (int c = 0; c < kChunks; ++c) d[c] = tag(q, p, c);
    if (q + 1 - q_sig > lag) publish();
  }
  while (q_sig < r.T) publish();
}

void consume(Ring& r, uint32_t q, uint32_t slot, uint32_t target) {
#ifdef PLANT_EARLY_READ
  target -= 1;
#endif
  if (!wait_for(r, r.full[slot], target)) return;
#ifdef PLANT_EARLY_RELEASE
  r.empty[slot].fetch_add(1, std::memory_order_release);
#endif
  for (uint32_t p = 0; p < r.NP; ++p) {
    const uint64_t* d = r.share(slot, p);
    for (int c = 0; c < kChunks; ++c)
      if (d[c] != tag(q, p, c)) r.mismatches.fetch_add(1);
  }
  // the kernels' consumers see K-iteration q + 1 full before releasing q
  if (r.lag >= 0 && q + 1 < r.T &&
      !wait_for(r, r.full[wsg::ring_slot(q + 1, r.P)], wsg::ring_full_target(q + 1, r.P, r.NP)))
    return;
#ifndef PLANT_EARLY_RELEASE
  r.empty[slot].fetch_add(1, std::memory_order_release);
#endif
}

void consumer_closed_form(Ring& r) {
  for (uint32_t q = 0; q < r.T && !r.abort.load(std::memory_order_relaxed); ++q)
    consume(r, q, wsg::ring_slot(q, r.P), wsg::ring_full_target(q, r.P, r.NP));
}

void consumer_incremental(Ring& r) {
  uint32_t slot = wsg::ring_slot(0, r.P), target = wsg::ring_full_target(0, r.P, r.NP);
  for (uint32_t q = 0; q < r.T && !r.abort.load(std::memory_order_relaxed); ++q) {
    if (slot != wsg::ring_slot(q, r.P) || target != wsg::ring_full_target(q, r.P, r.NP)) {
      r.mismatches.fetch_add(1);  // the two walks disagree
      return;
    }
    consume(r, q, slot, target);
    wsg::ring_advance(slot, target, r.P, r.NP);
  }
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 6 && argc != 7) {
    std::fprintf(stderr, "usage: %s P NP NC T WAIT_LIMIT_MS [LAG]\n", argv[0]);
    return 3;
  }
  const long P = std::atol(argv[1]), NP = std::atol(argv[2]), NC = std::atol(argv[3]);
  const long T = std::atol(argv[4]);
  const long long limit = std::atoll(argv[5]);
  if (P < 1 || P > 64 || NP < 1 || NP > 64 || NC < 1 || NC > 64 || T < 1 || limit < 1) return 3;
  const long lag = argc == 7 ? std::atol(argv[6]) : -1;
  // a consumer that looks one K-iteration ahead needs two slots at least
  if (lag < -1 || lag > 64 || (lag >= 0 && P < 2)) return 3;
  Ring r((uint32_t)P, (uint32_t)NP, (uint32_t)NC, (uint32_t)T, limit);
  r.lag = (int)lag;
  std::vector<std::thread> th;
  for (uint32_t p = 0; p < r.NP; ++p) th.emplace_back(lag >= 0 ? producer_deferred : producer, std::ref(r), p);
  for (uint32_t c = 0; c < r.NC; ++c)
    th.emplace_back((c % 2) ? consumer_incremental : consumer_closed_form, std::ref(r));
  for (auto& t : th) t.join();
  std::printf("P=%ld NP=%ld NC=%ld T=%ld lag=%ld timeouts=%d mismatches=%d\n", P, NP, NC, T, lag,
              r.timeouts.load(), r.mismatches.load());
  if (r.timeouts.load()) return 2;
  if (r.mismatches.load()) return 1;
  return 0;
}

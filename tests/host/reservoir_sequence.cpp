// CPU test of a reservoir's host call protocol (paper_2309_16743_amd/csrc/res_host.h,
// the code the library runs under each reservoir's mutex), built with the
// thread sanitizer: producer and consumer threads put and draw concurrently
// (some calls fail before they are ordered, as a failed HIP event call would),
// one thread ends reception part-way, and the work each call enqueues on the
// emulated ordering stream is recorded.  Checked afterwards: the recorded
// tickets are 0, 1, 2, ... in stream order (ticket order is execution order,
// failed calls take no ticket); replaying the recorded calls one by one in
// ticket order on a fresh state reproduces every call's kernel arguments
// (the host state is a function of the ticket sequence alone); N stays in
// [0, C], ring positions in [0, C); no put is ordered after reception ended.
// With -DPLANT_RACE one thread also reads N without the mutex, which the
// sanitizer must report (so that a clean run means the sanitizer ran).
#include <atomic>
#include <cstdio>
#include <mutex>
#include <random>
#include <thread>
#include <vector>

#include "res_host.h"

namespace {

struct Rec {
  int kind = 0;                  // 0 put, 1 draw, 2 end of reception
  int64_t arg = 0;               // k or b
  ot::PutCall put;
  ot::DrawCall draw;
};

struct Model {
  std::mutex mu;
  ot::ResSeq seq;
  std::vector<Rec> stream;       // the ordering stream: work in enqueue order
};

int put(Model& m, int64_t k, bool enter_fails) {
  std::lock_guard<std::mutex> lock(m.mu);
  const int st = ot::put_admit(m.seq);
  if (st != OT_OK) return st;
  if (enter_fails) return OT_E_HIP;
  Rec r;
  r.kind = 0;
  r.arg = k;
  r.put = ot::put_commit(m.seq, k);
  m.stream.push_back(r);
  return OT_OK;
}

int draw(Model& m, int64_t b, bool enter_fails) {
  std::lock_guard<std::mutex> lock(m.mu);
  int64_t drawn = 0;
  const int st = ot::draw_admit(m.seq, b, &drawn);
  if (st != OT_OK) return st;
  if (enter_fails) return OT_E_HIP;
  Rec r;
  r.kind = 1;
  r.arg = b;
  r.draw = ot::draw_commit(m.seq, drawn);
  m.stream.push_back(r);
  return OT_OK;
}

bool same(const ot::PutCall& a, const ot::PutCall& b) {
  return a.ticket == b.ticket && a.n_before == b.n_before && a.accepted == b.accepted && a.may_evict == b.may_evict &&
         a.free_head == b.free_head;
}
bool same(const ot::DrawCall& a, const ot::DrawCall& b) {
  return a.ticket == b.ticket && a.n_before == b.n_before && a.drawn == b.drawn && a.take == b.take &&
         a.occ_base == b.occ_base && a.free_tail == b.free_tail;
}

int run(int32_t policy) {
  const int64_t C = 64, T = 10;
  Model m;
  m.seq.policy = policy;
  m.seq.C = C;
  m.seq.T = T;
  std::atomic<int> calls{0};
  std::vector<std::thread> th;
  for (int p = 0; p < 6; ++p)
    th.emplace_back([&, p] {
      std::mt19937 g(1000 + p);
      for (int i = 0; i < 1500; ++i) {
        put(m, (int64_t)(g() % 9), g() % 50 == 0);
        calls.fetch_add(1);
      }
    });
  for (int c = 0; c < 4; ++c)
    th.emplace_back([&, c] {
      std::mt19937 g(2000 + c);
      for (int i = 0; i < 2500; ++i) {
        draw(m, 1 + (int64_t)(g() % 12), g() % 50 == 0);
        calls.fetch_add(1);
      }
    });
  th.emplace_back([&] {
    while (calls.load() < 9000) std::this_thread::yield();
    std::lock_guard<std::mutex> lock(m.mu);
    if (ot::end_commit(m.seq) == OT_OK) {
      Rec r;
      r.kind = 2;
      m.stream.push_back(r);
    }
  });
#ifdef PLANT_RACE
  th.emplace_back([&] {
    int64_t seen = 0;
    for (int i = 0; i < 20000; ++i) seen += m.seq.n_host;   // no mutex: a data race
    std::printf("planted read: %lld\n", (long long)seen);
  });
#endif
  for (auto& t : th) t.join();

  // replay in stream order on a fresh state
  ot::ResSeq q;
  q.policy = policy;
  q.C = C;
  q.T = T;
  uint64_t expect_ticket = 0;
  bool ended = false;
  int64_t puts = 0, draws = 0;
  for (size_t i = 0; i < m.stream.size(); ++i) {
    const Rec& r = m.stream[i];
    if (r.kind == 2) {
      if (ot::end_commit(q) != OT_OK) { std::printf("FAIL end of reception refused on replay\n"); return 1; }
      ended = true;
      continue;
    }
    if (r.kind == 0) {
      if (ended || ot::put_admit(q) != OT_OK) { std::printf("FAIL put ordered after reception ended\n"); return 1; }
      const ot::PutCall c = ot::put_commit(q, r.arg);
      if (c.ticket != expect_ticket || !same(c, r.put)) {
        std::printf("FAIL put %zu: ticket %llu (expected %llu), replay differs\n", i, (unsigned long long)r.put.ticket,
                    (unsigned long long)expect_ticket);
        return 1;
      }
      ++puts;
    } else {
      int64_t drawn = 0;
      if (ot::draw_admit(q, r.arg, &drawn) != OT_OK) { std::printf("FAIL draw %zu not admitted on replay\n", i); return 1; }
      const ot::DrawCall c = ot::draw_commit(q, drawn);
      if (c.ticket != expect_ticket || !same(c, r.draw)) {
        std::printf("FAIL draw %zu: ticket %llu (expected %llu), replay differs\n", i,
                    (unsigned long long)r.draw.ticket, (unsigned long long)expect_ticket);
        return 1;
      }
      ++draws;
    }
    ++expect_ticket;
    if (q.n_host < 0 || q.n_host > C || q.occ_base < 0 || q.occ_base >= C || q.free_head < 0 || q.free_head >= C) {
      std::printf("FAIL state out of range after record %zu\n", i);
      return 1;
    }
  }
  if (q.next_ticket != m.seq.next_ticket || q.n_host != m.seq.n_host) {
    std::printf("FAIL final state differs from the replay\n");
    return 1;
  }
  std::printf("policy %d: %lld puts, %lld draws ordered, tickets 0..%llu, reception %s, final N %lld\n", (int)policy,
              (long long)puts, (long long)draws, (unsigned long long)expect_ticket - 1, ended ? "ended" : "open",
              (long long)q.n_host);
  return 0;
}

}  // namespace

int main() {
  for (int32_t policy : {OT_POLICY_RESERVOIR, OT_POLICY_FIFO, OT_POLICY_FIRO})
    if (run(policy) != 0) return 1;
  std::printf("ok\n");
  return 0;
}

// ThreadSanitizer check of the library's host-side concurrency (built with g++
// -fsanitize=thread by tests/test_host_threads_tsan.py, no device involved):
//  - the CPU share's worker team (cpu_share, team_for): jobs submitted from several
//    host threads at once (the team serialises them), batches 1-8, thread counts 1-8,
//    while another thread flips the streamed-chunk count that sets the team's spin
//    policy; every result must equal the single-threaded bits;
//  - the pin team (PinTeam), which stages pageable weights into pinned buffers
//    (Sec. 4.2 hybrid pin || transfer): copies of 1-9 MiB split over its threads,
//    checked byte for byte, then a shutdown and a restart with another thread count.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <random>
#include <thread>
#include <vector>

#include "../../paper_2403_01164_amd/csrc/cpu_share.h"
#include "../../paper_2403_01164_amd/csrc/pin_team.h"

namespace {

int g_fail = 0;

void check(bool ok, const char* what) {
  if (!ok) {
    fprintf(stderr, "FAILED: %s\n", what);
    g_fail = 1;
  }
}

struct Problem {
  int B, K, N, dtype;
  std::vector<float> x;
  std::vector<uint16_t> W, bias;
  std::vector<float> ref;
};

Problem make(int B, int K, int N, int dtype, unsigned seed) {
  Problem p{B, K, N, dtype, {}, {}, {}, {}};
  std::mt19937 rng(seed);
  std::uniform_int_distribution<int> small(-3, 3);
  p.x.resize((size_t)B * K);
  for (auto& v : p.x) v = (float)small(rng) * 0.25f;
  // 16-bit weights: fp16 / bf16 encodings of small integers times 1/8 (exact in both)
  p.W.resize((size_t)N * K);
  p.bias.resize(N);
  auto enc = [&](float f) -> uint16_t {
    uint32_t u;
    memcpy(&u, &f, 4);
    if (dtype == 1) return (uint16_t)(u >> 16);
    // fp16 of a value with at most 3 significant bits and a small exponent
    const uint32_t sign = (u >> 16) & 0x8000u;
    if ((u & 0x7FFFFFFFu) == 0) return (uint16_t)sign;
    const int e = (int)((u >> 23) & 0xFF) - 127 + 15;
    return (uint16_t)(sign | ((uint32_t)e << 10) | ((u >> 13) & 0x3FFu));
  };
  for (auto& w : p.W) w = enc((float)small(rng) * 0.125f);
  for (auto& b : p.bias) b = enc((float)small(rng) * 0.125f);
  p.ref.resize((size_t)B * N);
  hg::cpu_share(p.x.data(), B, K, p.W.data(), dtype, p.bias.data(), 0, N, p.ref.data(), N, 1);
  return p;
}

}  // namespace

int main() {
  // ---- CPU-share worker team: concurrent callers ----
  std::vector<Problem> probs;
  for (int B = 1; B <= 8; ++B) probs.push_back(make(B, 520, 203, B & 1, 100u + B));
  std::atomic<bool> stop{false};
  std::thread flipper([&] {
    for (int i = 0; !stop.load(); ++i) {
      hg::team_streamed_chunks(i % 2 ? -1 : 1);
      std::this_thread::sleep_for(std::chrono::microseconds(50));
    }
  });
  std::vector<std::thread> callers;
  std::atomic<int> bad{0};
  for (int c = 0; c < 4; ++c) {
    callers.emplace_back([&, c] {
      for (int it = 0; it < 24; ++it) {
        const Problem& p = probs[(c * 3 + it) % probs.size()];
        const int threads = 1 + (c + it) % 8;
        std::vector<float> y((size_t)p.B * p.N, -1.f);
        hg::cpu_share(p.x.data(), p.B, p.K, p.W.data(), p.dtype, p.bias.data(), 0, p.N, y.data(), p.N, threads);
        if (memcmp(y.data(), p.ref.data(), y.size() * sizeof(float)) != 0) bad++;
        // a row range: rows [17, 150) land at y[b * 150 + r - 17]
        std::vector<float> z((size_t)p.B * 150, -1.f);
        hg::cpu_share(p.x.data(), p.B, p.K, p.W.data(), p.dtype, p.bias.data(), 17, 150, z.data(), 150, threads);
        for (int b = 0; b < p.B; ++b)
          if (memcmp(&z[(size_t)b * 150], &p.ref[(size_t)b * p.N + 17], 133 * sizeof(float)) != 0) bad++;
      }
    });
  }
  // team_for from another thread at the same time: each grain adds its index once
  std::thread other([&] {
    for (int it = 0; it < 40; ++it) {
      struct Acc {
        std::atomic<long long> sum{0};
      } acc;
      hg::team_for(1 + it % 8, 100, [](void* a, int g) { ((Acc*)a)->sum.fetch_add(g); }, &acc);
      if (acc.sum.load() != 4950) bad++;
    }
  });
  for (auto& t : callers) t.join();
  other.join();
  stop = true;
  flipper.join();
  check(bad.load() == 0, "worker team results");

  // ---- pin team ----
  std::mt19937 rng(7);
  for (int round = 0; round < 2; ++round) {
    hg::PinTeam team;
    check(team.start(round == 0 ? 4 : 3), "pin team start");
    std::vector<char> src(10 << 20), dst(10 << 20);
    for (size_t i = 0; i < src.size(); ++i) src[i] = (char)(i * 131 + round);
    for (int it = 0; it < 20; ++it) {
      const size_t n = (1 << 20) + rng() % (8 << 20), off = rng() % 4096;
      memset(dst.data(), 0x5A, dst.size());
      team.copy(dst.data() + off, src.data() + off, n);
      check(memcmp(dst.data() + off, src.data() + off, n) == 0, "pin team copy");
      check(off == 0 || dst[off - 1] == 0x5A, "pin team copy stays in bounds (front)");
      check(off + n >= dst.size() || dst[off + n] == 0x5A, "pin team copy stays in bounds (back)");
    }
    team.shutdown();
  }
  printf(g_fail ? "host thread check FAILED\n" : "host thread check ok\n");
  return g_fail;
}

// Host-only exercise of libonela's configuration, layout, selection-plan and
// per-step protocol checks (host_plan.cpp), built with the address and
// undefined-behaviour sanitizers by tests/test_sanitizers.py.  Exits non-zero
// on the first violated expectation; the sanitizers abort on their own.
#include <cstdio>
#include <cstdlib>
#include <random>

#include "../../paper_2609_12399_amd/csrc/host_plan.h"

using namespace onela;

static int failures = 0;
#define EXPECT(c)                                                          \
  do {                                                                     \
    if (!(c)) {                                                            \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__,   \
                   __LINE__, #c);                                          \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

static void configs() {
  const int Rs[] = {0, 1, 3, 65537};
  const int heads[][2] = {{16, 16}, {16, 32}, {2, 3}, {0, 4}, {4, 8}};
  const int dims[][2] = {{32, 32}, {64, 64}, {128, 128}, {128, 256}, {128, 512},
                         {256, 256}, {256, 512}, {100, 100}, {256, 128}, {0, 0}};
  const int beams[] = {0, 1, 512, 65536, 65537};
  const int steps[] = {0, 1, 8, 9};
  int ok = 0;
  for (int R : Rs)
    for (auto& h : heads)
      for (auto& d : dims)
        for (int W : beams)
          for (int T : steps)
            for (int io = 0; io < 3; ++io)
              for (int rk = 0; rk < 3; ++rk)
                for (int st = 0; st < 3; ++st) {
                  onela_config_t c{R, h[0], h[1], d[0], d[1], W, T, io, rk, st};
                  Shape s{};
                  const onela_status_t rc = shape_of(&c, &s);
                  EXPECT(rc == ONELA_OK || rc == ONELA_EINVAL);
                  if (rc != ONELA_OK) continue;
                  ++ok;
                  EXPECT(s.R >= 1 && s.HV % s.HK == 0 && decode_supported(s));
                  const Layout l = layout_of(s);
                  const size_t parts[] = {l.status, l.anc, l.s_frag, l.k, l.v, l.ab, l.d, l.ds};
                  size_t sum = l.anc;  // the ancestry index is double-buffered
                  for (size_t x : parts) {
                    EXPECT(x % 256 == 0);
                    sum += x;
                  }
                  EXPECT(sum == l.total);
                  EXPECT(!s.borrow || (l.k == 0 && l.v == 0 && l.ab == 0));
                  EXPECT(s.delta == (l.d > 0));
                  EXPECT(prefill_chunked_workspace_bytes(s, 0) % 256 == 0);
                  EXPECT(prefill_chunked_workspace_bytes(s, 65) >=
                         prefill_chunked_workspace_bytes(s, 64));
                }
  EXPECT(ok > 0);
  EXPECT(shape_of(nullptr, nullptr) == ONELA_EINVAL);
}

static void select_plans() {
  const int Rs[] = {0, 1, 2, 64, 65, 65536, 65537};
  const int Ps[] = {0, 1, 3, 512, 1023, 4096, 65536};
  const int Vs[] = {0, 1, 5, 2047, 8192, 16385};
  const int Ws[] = {0, 1, 7, 64, 512, 1024, 4096, 4097};
  for (int R : Rs)
    for (int P : Ps)
      for (int V : Vs)
        for (int W : Ws) {
          SelectPlan plan{};
          const onela_status_t rc = check_select(R, P, V, W, &plan);
          const unsigned long long N = (unsigned long long)(P > 0 ? P : 0) * (V > 0 ? V : 0);
          if (R < 1 || R > 65536 || P < 1 || V < 1 || W < 1 || (unsigned long long)W > N ||
              W > kSelectMaxWidth || N > kSelectMaxCandidates) {
            EXPECT(rc == ONELA_EINVAL);
            continue;
          }
          EXPECT(rc == ONELA_OK);
          // the control block and the one-pass summary region come first in
          // every plan, and nothing else is placed there
          const size_t head = kSelectCtlBytes + kSelectSummaryBytes;
          EXPECT(plan.total % 256 == 0 && plan.total >= head);
          EXPECT(plan.cap >= unsigned(W) && (plan.cap & (plan.cap - 1)) == 0);
          if (plan.two_pass) {
            EXPECT(plan.seg_off == head);
            EXPECT(plan.seg_off < plan.bound_off && plan.bound_off < plan.slot_off &&
                   plan.slot_off < plan.cnt_off && plan.cnt_off < plan.total);
            EXPECT(plan.bound_off - plan.seg_off >= size_t(R) * plan.nseg * 16);
            EXPECT(plan.nseg == plan.nchunks * 8u);
            EXPECT(uint64_t(plan.nchunks) * kSelectChunk >= N);
          } else {
            EXPECT(plan.stages >= 0 && plan.stages <= kSelectMaxStages);
            for (int b = 0; b < 2; ++b)
              EXPECT(plan.pair_off[b] >= head && plan.count_off[b] <= plan.total);
          }
        }
}

// The protocol as onela_api.cpp drives it: a random walk of calls, each
// applied to the state only when its check passes.
static void protocol_walk() {
  std::mt19937 rng(7);
  onela_config_t c{2, 4, 8, 128, 128, 64, 4, ONELA_BF16, ONELA_RECORD_INPUTS, ONELA_RECORDS_COPY};
  Shape s{};
  EXPECT(shape_of(&c, &s) == ONELA_OK);
  alignas(16) static char buf[64];
  const void* ptrs[] = {nullptr, buf, buf + 4, buf + 1, buf + 16};
  Protocol pr;
  for (int it = 0; it < 200000; ++it) {
    if (rng() % 97 == 0) pr = Protocol{};  // reset
    const int call = int(rng() % 4);
    const int step = int(rng() % 7) - 1;
    const int width = int(rng() % 70) - 2;
    auto P = [&]() { return ptrs[rng() % 5]; };
    const Protocol before = pr;
    onela_status_t rc;
    switch (call) {
      case 0:
        rc = check_resolve(s, pr, step, width, P(), P());
        if (rc == ONELA_OK) {
          EXPECT(step >= 0 && step < s.tmax && width >= 1 && width <= s.wmax);
          pr.widths[step] = width;
          pr.resolved = step;
        }
        break;
      case 1:
        rc = check_append(pr, step, P(), P(), P(), P());
        if (rc == ONELA_OK) pr.appended = step;
        break;
      case 2:
        rc = check_decode(pr, step, P(), P());
        if (rc == ONELA_OK) EXPECT(pr.widths[step] >= 1);
        break;
      default:
        rc = check_fused(s, pr, step, width, P(), P(), P(), P(), P(), P(), P(), P());
        if (rc == ONELA_OK) {
          pr.widths[step] = width;
          pr.resolved = pr.appended = step;
        }
    }
    EXPECT(rc == ONELA_OK || rc == ONELA_EINVAL || rc == ONELA_ESTEP || rc == ONELA_ECAPACITY);
    if (rc != ONELA_OK && call != 2) {
      EXPECT(pr.resolved == before.resolved && pr.appended == before.appended);
    }
    EXPECT(pr.resolved >= -1 && pr.resolved < s.tmax);
    EXPECT(pr.appended <= pr.resolved && pr.appended >= pr.resolved - 1);
  }
}

int main() {
  configs();
  select_plans();
  protocol_walk();
  if (failures) {
    std::fprintf(stderr, "%d expectation(s) failed\n", failures);
    return 1;
  }
  std::printf("host plan checks: ok\n");
  return 0;
}

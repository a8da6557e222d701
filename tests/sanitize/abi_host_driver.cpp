// Drives the host side of libtfg's C ABI (argument checks, size queries,
// status strings) with no GPU: every call below either only computes sizes
// or fails its checks before touching device memory or the HIP runtime. Built
// with AddressSanitizer and UndefinedBehaviorSanitizer on the host code by
// tests/test_sanitize.py (the device code is compiled as usual).
#include <cstdio>
#include <cstring>

#include "../../include/tfg.h"

static int failures = 0;
#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                            \
    }                                                                        \
  } while (0)

int main() {
  void* fake = reinterpret_cast<void*>(0x1000);  // never dereferenced
  tfg_graph* h = nullptr;
  size_t b = 0, s = 0;
  for (int st = 0; st < 8; ++st) CHECK(std::strlen(tfg_status_string(st)) > 0);
  CHECK(tfg_abi_version() == TFG_ABI_VERSION);
  // size queries over a range of sizes, parts and widths
  const int64_t sizes[] = {0, 1, 7, 1000, 123457, (int64_t(1) << 31) - (int64_t(1) << 20) - 1};
  for (int64_t E : sizes)
    for (int64_t N : {int64_t(1), int64_t(10), int64_t(4097), int64_t(232965)})
      for (int parts : {0, 1, 3, 16}) {
        const int rc = tfg_graph_bytes(E, N, N, 0, parts, &b, &s);
        CHECK(rc == TFG_OK || rc == TFG_ERR_TOO_LARGE);
        CHECK(tfg_gcn_norm_ws_bytes(E, N, 1, nullptr) > 0 || E + N >= (int64_t(1) << 31));
        for (int64_t F : {int64_t(1), int64_t(64), int64_t(128)})
          for (int red = 0; red < 3; ++red) (void)tfg_aggregate_ws_bytes(E, N, N, F, red, nullptr);
        (void)tfg_segment_pool_ws_bytes(E, N);
        (void)tfg_segment_softmax_ws_bytes(E, 8, N, nullptr);
        (void)tfg_gat_edge_scores_ws_bytes(N, 8);
        (void)tfg_batch_graphs_ws_bytes(N);
      }
  CHECK(tfg_graph_bytes(-1, 100, 100, 0, 0, &b, &s) == TFG_ERR_INVALID_ARG);
  CHECK(tfg_graph_bytes(int64_t(1) << 31, 10, 10, 0, 0, &b, &s) == TFG_ERR_TOO_LARGE);
  // graph creation: NULL handle, bad index type, loops on a rectangle, small or misaligned buffers
  CHECK(tfg_graph_create(fake, 0, 10, 5, 5, 0, 0, fake, 1 << 20, fake, 1 << 20, nullptr, nullptr) == 1);
  CHECK(tfg_graph_create(fake, 7, 10, 5, 5, 0, 0, fake, 1 << 20, fake, 1 << 20, nullptr, &h) == 1);
  CHECK(tfg_graph_create(fake, 0, 10, 4, 5, 1, 0, fake, 1 << 20, fake, 1 << 20, nullptr, &h) == 1);
  CHECK(tfg_graph_create(fake, 0, 10, 5, 5, 0, 0, fake, 16, fake, 1 << 20, nullptr, &h) == 5);
  CHECK(std::strstr(tfg_last_error(), "too small") != nullptr);
  CHECK(tfg_graph_create(fake, 0, 10, 5, 5, 0, 0, reinterpret_cast<void*>(0x1080), 1 << 20, fake,
                         1 << 20, nullptr, &h) == 5);
  CHECK(tfg_graph_create_transposed(fake, 9, 10, 5, 5, 0, 0, fake, 1 << 20, fake, 1 << 20,
                                    nullptr, &h) == 1);
  // aggregation: bad reduce, heads, ldx, orders, workspace, sizes; the no-allocation form
  float* ff = static_cast<float*>(fake);
  CHECK(tfg_aggregate(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 8, 5, 3, nullptr, ff, nullptr, fake,
                      1 << 30, nullptr) == 1);
  CHECK(tfg_aggregate(fake, 0, 10, ff, 3, 0, ff, 5, 8, 8, 5, 0, nullptr, ff, nullptr, fake,
                      1 << 30, nullptr) == 1);
  CHECK(tfg_aggregate(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 4, 5, 0, nullptr, ff, nullptr, fake,
                      1 << 30, nullptr) == 1);
  CHECK(tfg_aggregate(fake, 0, 10, ff, 1, 1, ff, 5, 8, 8, 5, 0, nullptr, ff, nullptr, fake,
                      1 << 30, nullptr) == 1);
  CHECK(tfg_aggregate(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 8, 5, 0, nullptr, ff, nullptr, fake, 8,
                      nullptr) == 5);
  CHECK(tfg_aggregate(fake, 0, -1, nullptr, 1, 0, ff, 5, 8, 8, 5, 0, nullptr, ff, nullptr, fake,
                      1 << 30, nullptr) == 1);
  CHECK(tfg_aggregate(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 8, int64_t(1) << 31, 0, nullptr, ff,
                      nullptr, fake, 1 << 30, nullptr) == 4);
  CHECK(tfg_aggregate_noalloc(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 8, 5, 0, nullptr, ff, nullptr,
                              nullptr) == 1);  // needs a graph handle
  CHECK(tfg_aggregate_noalloc(fake, 0, 10, nullptr, 1, 0, ff, 5, 8, 8, 5, 7, nullptr, ff, nullptr,
                              nullptr) == 1);
  // pooling, softmax, scores, backward, reorder, attention, propagation, batching
  CHECK(tfg_segment_pool(ff, 10, 4, 4, fake, 0, 3, 5, ff, nullptr, 1, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_segment_pool(ff, 10, 4, 2, fake, 0, 3, 0, ff, nullptr, 1, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_segment_softmax(ff, 10, 2, fake, 0, 5, nullptr, ff, ff, fake, 1 << 30, nullptr) == 1);
  CHECK(tfg_gat_edge_scores(fake, 0, 10, ff, 5, 0, 4, ff, ff, 0.2f, ff, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_aggregate_backward(nullptr, nullptr, nullptr, 1, 0, ff, 8, ff, 8, 0, nullptr, ff,
                               nullptr, 0, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_aggregate_backward_ws_bytes(nullptr, nullptr, 8, 1, 0, 0, 0) == 0);
  CHECK(tfg_edge_reorder(nullptr, nullptr, ff, 1, ff, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_segment_softmax_backward(ff, ff, 10, 0, fake, 0, 5, nullptr, ff, fake, 1 << 30,
                                     nullptr) == 1);
  CHECK(tfg_gat_aggregate(nullptr, ff, 8, 16, ff, ff, 0.2f, ff, nullptr, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_propagate(nullptr, nullptr, 0, ff, 8, 8, 2, 0.0f, nullptr, 0, ff, fake, 1 << 20,
                      nullptr) == 1);
  CHECK(tfg_batch_graphs(-1, fake, fake, fake, 0, 0, 0, fake, fake, nullptr, nullptr, 1, fake,
                         1 << 20, nullptr) == 1);
  CHECK(tfg_gat_graph_scores(nullptr, ff, 8, 16, ff, ff, 0.2f, ff, 1, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_segment_softmax_graph(nullptr, ff, 8, 1, ff, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_segment_softmax_graph_backward(nullptr, ff, ff, 8, 1, ff, fake, 1 << 20, nullptr) == 1);
  CHECK(tfg_gat_graph_scores_ws_bytes(nullptr, 8) == 0);
  CHECK(tfg_segment_softmax_graph_ws_bytes(nullptr, 8) == 0);
  int64_t nb = 0, ne = 0;
  CHECK(tfg_batch_graphs_totals(-1, fake, fake, 0, fake, 1 << 20, nullptr, &nb, &ne) == 1);
  CHECK(tfg_batch_graphs_totals(4, fake, fake, 0, fake, 1 << 20, nullptr, nullptr, &ne) == 1);
  CHECK(tfg_batch_graphs_totals(0, nullptr, nullptr, 0, fake, 1 << 20, nullptr, &nb, &ne) == 0 &&
        nb == 0 && ne == 0);
  CHECK(tfg_graph_destroy(nullptr) == 0 || tfg_graph_destroy(nullptr) == 1);
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("abi host driver ok\n");
  return 0;
}

// Exercises the C ABI's host code (include/bifattn.h) under AddressSanitizer
// and UndefinedBehaviorSanitizer, linked with launch stand-ins and run
// without a GPU: every argument check, dimension limits up to the largest
// values the types hold, the allocation-free entry point's size check, the
// status strings, and the many-row kernels' XCD order of work-groups. Exit status 0 when every call returns what the header
// documents.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include <vector>

#include "bifattn.h"
#include "bifattn_internal.h"

static int failures = 0;
#define EXPECT(call, ...)                                                              \
  do {                                                                                 \
    const int got_ = (int)(call);                                                      \
    bool ok_ = false;                                                                  \
    for (int want_ : {__VA_ARGS__}) ok_ |= got_ == want_;                              \
    if (!ok_) {                                                                        \
      std::fprintf(stderr, "%s:%d: %s returned %d\n", __FILE__, __LINE__, #call, got_); \
      ++failures;                                                                      \
    }                                                                                  \
  } while (0)

static bifattn_dims_t dims(int b, int h, int g, int d, int m_c, int m_d, float scale = 0.f,
                           int n = 1, int kv = BIFATTN_KV_BF16, int path = BIFATTN_PATH_AUTO) {
  bifattn_dims_t x;
  std::memset(&x, 0, sizeof x);
  x.b = b;
  x.h = h;
  x.g = g;
  x.d = d;
  x.m_c = m_c;
  x.m_d_max = m_d;
  x.scale = scale;
  x.n = n;
  x.kv_type = kv;
  x.path = path;
  return x;
}

// The many-row context kernels' dispatch-id mapping: a permutation of the
// logical ids, every row block of each of the first kXcds * (chunks / kXcds)
// chunks on one XCD (dispatch id % kXcds), and, when each XCD's share of ids
// holds whole chunks, the plain strided order (id % kXcds) * share + id / kXcds.
static void check_xcd_mapping() {
  using bifattn::kXcds;
  using bifattn::xcd_logical;
  for (int chunks = 1; chunks <= 70; ++chunks)
    for (int rows = 1; rows <= 20; ++rows) {
      const int n = chunks * rows, whole = kXcds * (chunks / kXcds);
      std::vector<int> seen(n, 0), xcd(chunks, -1);
      for (int bid = 0; bid < n; ++bid) {
        const int l = xcd_logical(bid, chunks, rows);
        if (l < 0 || l >= n || seen[l]++) {
          std::fprintf(stderr, "xcd mapping not a permutation: chunks %d rows %d id %d\n", chunks,
                       rows, bid);
          ++failures;
          return;
        }
        const int c = l / rows;
        if (c < whole) {
          if (xcd[c] == -1) xcd[c] = bid % kXcds;
          if (xcd[c] != bid % kXcds) {
            std::fprintf(stderr, "chunk %d split over XCDs: chunks %d rows %d\n", c, chunks, rows);
            ++failures;
          }
        }
        const int share = n / kXcds;
        if (n % kXcds == 0 && share % rows == 0 && l != (bid % kXcds) * share + bid / kXcds) {
          std::fprintf(stderr, "xcd mapping not the strided order: chunks %d rows %d\n", chunks,
                       rows);
          ++failures;
        }
      }
    }
}

int main() {
  check_xcd_mapping();
  const int BIG = std::numeric_limits<int32_t>::max();
  bifattn_plan_t plan = reinterpret_cast<bifattn_plan_t>(1);
  EXPECT(bifattn_plan_create(nullptr, &plan), BIFATTN_EINVAL);
  if (plan != nullptr) { std::fprintf(stderr, "plan not cleared\n"); ++failures; }
  bifattn_dims_t bad[] = {
      dims(0, 4, 4, 64, 128, 16),        dims(4, 4, 3, 64, 128, 16),
      dims(4, 4, 4, 64, 0, 16),          dims(4, 4, 4, 64, 128, -1),
      dims(4, 4, 4, 64, 128, 16, NAN),   dims(4, 4, 4, 64, 128, 16, INFINITY),
      dims(4, 4, 4, 64, 128, 16, 0, -1), dims(4, 4, 4, 64, 128, 16, 0, 1, 7),
      dims(4, 4, 4, 64, 128, 16, 0, 1, 0, 9),
      dims(BIG, BIG, BIG, 128, BIG, BIG), dims(BIG, 64, 1, 128, 16, 16),
      dims(1 << 20, 1 << 10, 1 << 10, 128, 1 << 20, 1 << 20),
      dims(1, 64, 1, 128, BIG, BIG, 0, BIG),
  };
  for (const auto& x : bad) {
    EXPECT(bifattn_plan_create(&x, &plan), BIFATTN_EINVAL, BIFATTN_EUNSUPPORTED);
    EXPECT(bifattn_decode_noalloc(&x, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr, nullptr, nullptr),
           BIFATTN_EINVAL, BIFATTN_EUNSUPPORTED);
  }
  const bifattn_dims_t unsupported[] = {
      dims(4, 4, 4, 96, 128, 16), dims(4, 128, 1, 128, 128, 16), dims(4, 32, 1, 128, 128, 16, 0, 4),
      dims(2, 4, 1, 128, (1 << 23), 0),
      dims(2, 4, 1, 128, (1 << 25), 0, 0, 1, BIFATTN_KV_INT4),  // 2^31 bytes of int4 rows
  };
  for (const auto& x : unsupported) EXPECT(bifattn_plan_create(&x, &plan), BIFATTN_EUNSUPPORTED);
  // Valid dims: the plan needs a device (none here, or a real one).
  const bifattn_dims_t good[] = {
      dims(32, 32, 32, 128, 8192, 512), dims(128, 32, 1, 128, 16384, 512),
      dims(256, 32, 8, 128, 32768, 1024), dims(4, 4, 4, 64, 128, 16, 0, 1, 0, 2),
      dims(32, 32, 32, 128, 8192, 512, -0.1f, 4, BIFATTN_KV_FP8_E4M3, BIFATTN_PATH_BIFURCATED),
      dims(1, 1, 1, 64, 1, 0, 0, 1, BIFATTN_KV_INT8, BIFATTN_PATH_STANDARD),
      dims(32, 32, 32, 128, 8192, 512, 0, 1, BIFATTN_KV_INT4, BIFATTN_PATH_AUTO),
      dims(2, 4, 1, 128, (1 << 23), 0, 0, 1, BIFATTN_KV_INT4),  // 2^29 bytes of int4 rows
  };
  for (const auto& x : good) {
    plan = nullptr;
    const bifattn_status_t st = bifattn_plan_create(&x, &plan);
    EXPECT(st, BIFATTN_OK, BIFATTN_EHIP);
    if (st == BIFATTN_OK) EXPECT(bifattn_plan_destroy(plan), BIFATTN_OK);
    // the allocation-free entry point: argument checks or no device
    EXPECT(bifattn_decode_noalloc(&x, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr, nullptr, nullptr),
           BIFATTN_EINVAL, BIFATTN_EHIP);
  }
  // workspace beyond the fixed scratch: refused before any HIP call
  const bifattn_dims_t huge = dims(1024, 64, 1, 128, 65536, 1024);
  alignas(16) char dummy[256];
  const int32_t* lens = reinterpret_cast<const int32_t*>(dummy);
  EXPECT(bifattn_decode_noalloc(&huge, dummy, dummy, dummy, dummy, dummy, lens, nullptr, nullptr,
                                reinterpret_cast<float*>(dummy), nullptr),
         BIFATTN_ESCRATCH);
  // null handles
  EXPECT(bifattn_plan_destroy(nullptr), BIFATTN_OK);
  EXPECT(bifattn_plan_get_info(nullptr, nullptr), BIFATTN_EINVAL);
  EXPECT(bifattn_decode(nullptr, dummy, dummy, dummy, dummy, dummy, nullptr,
                        reinterpret_cast<float*>(dummy), nullptr),
         BIFATTN_EINVAL);
  EXPECT(bifattn_decode_replicated(nullptr, dummy, dummy, dummy, nullptr,
                                   reinterpret_cast<float*>(dummy), nullptr),
         BIFATTN_EINVAL);
  EXPECT(bifattn_append_kv(nullptr, dummy, dummy, dummy, dummy, nullptr, nullptr), BIFATTN_EINVAL);
  EXPECT(bifattn_plan_status(nullptr, nullptr), BIFATTN_EINVAL);
  EXPECT(bifattn_plan_set_timing(nullptr, BIFATTN_KERNEL_CALL, 1), BIFATTN_EINVAL);
  int32_t calls = 0;
  double ms = 0.0;
  EXPECT(bifattn_plan_read_timing(nullptr, &calls, &ms), BIFATTN_EINVAL);
  for (int s = -9; s <= 1; ++s) {
    const char* text = bifattn_status_string(static_cast<bifattn_status_t>(s));
    if (!text || !*text) {
      std::fprintf(stderr, "empty status string for %d\n", s);
      ++failures;
    }
  }
  EXPECT(bifattn_version(), BIFATTN_VERSION);
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("ABI driver: all checks passed\n");
  return 0;
}

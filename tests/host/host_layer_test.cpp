// Drives every entry point of the C ABI (include/twinkv.h) through the host layer with the
// kernel launchers stubbed out (stub_launchers.cpp): valid batches of several shapes (ragged
// lengths, empty sequences, strided keys, both key types and head dimensions) whose buffers
// are exactly as large as the ABI says, and invalid arguments whose return codes are checked.
// Built with AddressSanitizer and UndefinedBehaviorSanitizer: any out-of-range access of the
// host layer or of a range it hands to a kernel aborts the run.  Prints "host layer ok".
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <new>
#include <vector>

#include "twinkv.h"
#include "twinkv_internal.h"

namespace stub {
extern int64_t g_launches;
}

namespace {

int g_fail = 0;
#define EXPECT(cond)                                                          \
  do {                                                                        \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++g_fail;                                                               \
    }                                                                         \
  } while (0)

// Host memory standing in for device buffers: exactly the requested bytes (one for an empty
// range), 256-byte aligned, so that the sanitizer reports any access past the end.
struct Exact {
  std::vector<unsigned char*> owned;
  void* get(int64_t bytes) {
    unsigned char* p =
        new (std::align_val_t(256)) unsigned char[bytes > 0 ? (size_t)bytes : 1]();
    owned.push_back(p);
    return p;
  }
  ~Exact() {
    for (auto* p : owned) ::operator delete[](p, std::align_val_t(256));
  }
};

struct Shape {
  int n_heads, d, dtype;
  std::vector<int64_t> lens;
  int64_t tok_pad;  // extra elements per token (strided keys)
};

void run_shape(const Shape& sh) {
  Exact mem;
  const int H = sh.n_heads, d = sh.d, dt = sh.dtype, n_seqs = (int)sh.lens.size();
  std::vector<int64_t> cu(n_seqs + 1, 0);
  for (int s = 0; s < n_seqs; ++s) cu[s + 1] = cu[s] + sh.lens[s];
  const int64_t T = cu[n_seqs];
  const int64_t esz = dt == TWINKV_F32 ? 4 : 2;
  const int64_t ts = d + sh.tok_pad, hs = T * ts + (sh.tok_pad ? 8 : 0);
  // keys: exactly up to the last element of the last head
  const int64_t key_bytes = T > 0 ? esz * ((H - 1) * hs + (T - 1) * ts + d) : esz;
  // 16-byte alignment of the key pointer: new[] gives at least 16
  void* keys = mem.get(key_bytes);
  std::vector<int64_t> budget(n_seqs), cap(n_seqs);
  for (int s = 0; s < n_seqs; ++s) {
    budget[s] = sh.lens[s] / 2;
    cap[s] = sh.lens[s] - sh.lens[s] / 3;
  }
  const int64_t nt = (int64_t)H * T;
  void* ret = mem.get(nt);
  void* ret_out = mem.get(nt);
  float* fa = static_cast<float*>(mem.get(4 * nt));
  int32_t* ia = static_cast<int32_t*>(mem.get(4 * nt));
  float* fr = static_cast<float*>(mem.get(4 * nt));
  int32_t* ir = static_cast<int32_t*>(mem.get(4 * nt));
  int32_t* status = static_cast<int32_t*>(mem.get(4 * (int64_t)H * n_seqs));
  int32_t* stats = static_cast<int32_t*>(mem.get(16 * (int64_t)H * n_seqs));
  const int64_t* c = cu.data();

  for (int op : {TWINKV_OP_NN_SCORES, TWINKV_OP_REPAIR, TWINKV_OP_REPAIR_FROM_SCORES,
                 TWINKV_OP_TWIN_COUNTS, TWINKV_OP_SCORE_EVICT, TWINKV_OP_COMPACT}) {
    const int64_t wb = twinkv_workspace_bytes(op, dt, d, H, n_seqs, c);
    EXPECT(wb > 0);
    void* ws = mem.get(wb);
    int rc = -1;
    switch (op) {
      case TWINKV_OP_NN_SCORES:
        rc = twinkv_nn_scores(keys, dt, d, H, n_seqs, c, hs, ts, (uint8_t*)ret, 32, fa, ia, fr, ir,
                              status, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        rc = twinkv_nn_scores(keys, dt, d, H, n_seqs, c, hs, ts, nullptr, 0, fa, nullptr, nullptr,
                              nullptr, nullptr, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        EXPECT(twinkv_nn_scores(keys, dt, d, H, n_seqs, c, hs, ts, (uint8_t*)ret, 32, fa, ia, fr,
                                ir, status, ws, wb - 1, nullptr) == TWINKV_E_WORKSPACE);
        break;
      case TWINKV_OP_REPAIR:
        for (int all = 0; all < 2; ++all) {
          rc = twinkv_repair(keys, dt, d, H, n_seqs, c, hs, ts, (uint8_t*)ret, (uint8_t*)ret_out,
                             budget.data(), 0.9f, 32, 4, 16, stats, all ? fa : nullptr,
                             all ? ia : nullptr, all ? fr : nullptr, all ? ir : nullptr, ws, wb,
                             nullptr);
          EXPECT(rc == TWINKV_OK);
        }
        EXPECT(twinkv_repair(keys, dt, d, H, n_seqs, c, hs, ts, (uint8_t*)ret, (uint8_t*)ret_out,
                             budget.data(), 0.9f, -1, 4, 16, stats, nullptr, nullptr, nullptr,
                             nullptr, ws, wb, nullptr) == TWINKV_E_ARG);
        break;
      case TWINKV_OP_REPAIR_FROM_SCORES:
        rc = twinkv_repair_from_scores(fr, (uint8_t*)ret, (uint8_t*)ret_out, H, n_seqs, c,
                                       budget.data(), 0.9f, 4, 16, stats, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        rc = twinkv_select_topk(fr, H, n_seqs, c, budget.data(), 4, 16, (uint8_t*)ret_out, stats,
                                ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        {
          const float taus[3] = {0.8f, 0.9f, 0.95f};
          int32_t* prev = static_cast<int32_t*>(mem.get(4 * 3 * (int64_t)H * n_seqs));
          rc = twinkv_prevalence(fa, H, n_seqs, c, taus, 3, prev, ws, wb, nullptr);
          EXPECT(rc == TWINKV_OK);
        }
        break;
      case TWINKV_OP_TWIN_COUNTS:
        rc = twinkv_twin_counts(keys, dt, d, H, n_seqs, c, hs, ts, 0.9f, 32, ia, status, ws, wb,
                                nullptr);
        EXPECT(rc == TWINKV_OK);
        break;
      case TWINKV_OP_SCORE_EVICT:
        rc = twinkv_score_evict(keys, dt, d, H, n_seqs, c, hs, ts, budget.data(), 0.9f, 32, 4, 16,
                                (uint8_t*)ret_out, ia, fr, stats, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        break;
      case TWINKV_OP_COMPACT: {
        int64_t C = 0;
        for (int s = 0; s < n_seqs; ++s) C += cap[s];
        void* kout = mem.get(esz * d * H * C);
        void* vout = mem.get(esz * d * H * C);
        int32_t* pos = static_cast<int32_t*>(mem.get(4 * H * C));
        rc = twinkv_compact(keys, keys, dt, d, H, n_seqs, c, hs, ts, hs, ts, (uint8_t*)ret,
                            cap.data(), kout, vout, pos, stats, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        rc = twinkv_compact(keys, nullptr, dt, d, H, n_seqs, c, hs, ts, 0, 0, (uint8_t*)ret,
                            cap.data(), kout, nullptr, nullptr, stats, ws, wb, nullptr);
        EXPECT(rc == TWINKV_OK);
        break;
      }
    }
  }
  // nested retained sets
  for (int want_all = 0; want_all < 2; ++want_all) {
    const int L = 3;
    const int64_t wb = twinkv_levels_workspace_bytes(dt, d, H, n_seqs, c, L, want_all);
    EXPECT(wb > 0);
    void* ws = mem.get(wb);
    float* bl = static_cast<float*>(mem.get(4 * nt * L));
    int32_t* al = static_cast<int32_t*>(mem.get(4 * nt * L));
    const int rc = twinkv_nn_scores_levels(keys, dt, d, H, n_seqs, c, hs, ts, (uint8_t*)ret, L, 32,
                                           want_all ? fa : nullptr, want_all ? ia : nullptr, bl,
                                           al, status, ws, wb, nullptr);
    EXPECT(rc == TWINKV_OK);
  }
  // the variant without a workspace: its table goes to a caller-supplied region here
  {
    const size_t cap_bytes = sizeof(twinkv::SeqInfo) * (size_t)n_seqs;
    void* table = mem.get((int64_t)cap_bytes);
    const int rc = twinkv::repair_from_scores_into(fr, (uint8_t*)ret, (uint8_t*)ret_out, H, n_seqs,
                                                   c, budget.data(), 0.9f, 4, 16, stats, table,
                                                   cap_bytes, nullptr, nullptr);
    EXPECT(rc == TWINKV_OK);
    if (n_seqs > 1)
      EXPECT(twinkv::repair_from_scores_into(fr, (uint8_t*)ret, (uint8_t*)ret_out, H, n_seqs, c,
                                             budget.data(), 0.9f, 4, 16, stats, table,
                                             cap_bytes - 1, nullptr, nullptr) == TWINKV_E_CAPACITY);
  }
}

void invalid_arguments() {
  Exact mem;
  const int64_t cu[3] = {0, 50, 120};
  const int64_t bad_cu[3] = {0, 50, 40};
  const int64_t budget[2] = {10, 20};
  const int64_t big_budget[2] = {10, 71};
  void* keys = mem.get(2 * 2 * 120 * 64);
  void* m = mem.get(2 * 120);
  float* f = static_cast<float*>(mem.get(4 * 2 * 120));
  int32_t* st = static_cast<int32_t*>(mem.get(16 * 4));
  void* ws = mem.get(1 << 20);
  EXPECT(twinkv_workspace_bytes(9, 0, 64, 2, 2, cu) == -TWINKV_E_ARG);
  EXPECT(twinkv_workspace_bytes(0, 0, 96, 2, 2, cu) == -TWINKV_E_UNSUPPORTED);
  EXPECT(twinkv_workspace_bytes(0, 0, 64, 2, 2, bad_cu) == -TWINKV_E_ARG);
  EXPECT(twinkv_workspace_bytes(0, 0, 64, 2, 2, nullptr) == -TWINKV_E_NULL);
  EXPECT(twinkv_workspace_bytes(0, 0, 64, 0, 2, cu) == -TWINKV_E_ARG);
  EXPECT(twinkv_nn_scores(keys, 0, 64, 2, 2, bad_cu, 120 * 64, 64, nullptr, 32, f, nullptr,
                          nullptr, nullptr, nullptr, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_nn_scores(keys, 0, 64, 2, 2, cu, 120 * 64, 60, nullptr, 32, f, nullptr, nullptr,
                          nullptr, nullptr, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_nn_scores((char*)keys + 2, 0, 64, 2, 2, cu, 120 * 64, 64, nullptr, 32, f, nullptr,
                          nullptr, nullptr, nullptr, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_repair(keys, 0, 64, 2, 2, cu, 120 * 64, 64, (uint8_t*)m, (uint8_t*)m, big_budget,
                       0.9f, 32, 4, 4, st, nullptr, nullptr, nullptr, nullptr, ws, 1 << 20,
                       nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_repair(keys, 0, 64, 2, 2, cu, 120 * 64, 64, (uint8_t*)m, (uint8_t*)m, budget,
                       INFINITY, 32, 4, 4, st, nullptr, nullptr, nullptr, nullptr, ws, 1 << 20,
                       nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_repair_from_scores(nullptr, (uint8_t*)m, (uint8_t*)m, 2, 2, cu, budget, 0.9f, 4, 4,
                                   st, ws, 1 << 20, nullptr) == TWINKV_E_NULL);
  const float taus[40] = {0.5f};
  EXPECT(twinkv_prevalence(f, 2, 2, cu, taus, 40, st, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  EXPECT(twinkv_nn_scores_levels(keys, 0, 64, 2, 2, cu, 120 * 64, 64, (uint8_t*)m, 5, 32, nullptr,
                                 nullptr, f, nullptr, nullptr, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  const int64_t cap_bad[2] = {51, 0};
  EXPECT(twinkv_compact(keys, nullptr, 0, 64, 2, 2, cu, 120 * 64, 64, 0, 0, (uint8_t*)m, cap_bad,
                        ws, nullptr, nullptr, st, ws, 1 << 20, nullptr) == TWINKV_E_ARG);
  for (int code = 0; code <= 7; ++code) EXPECT(twinkv_status_string(code) != nullptr);
  EXPECT(twinkv_version() == 100);
}

}  // namespace

int main() {
  const std::vector<Shape> shapes = {
      {1, 64, TWINKV_F32, {512}, 0},
      {3, 128, TWINKV_BF16, {700, 0, 1, 4097, 33}, 0},
      {2, 64, TWINKV_BF16, {0, 0, 5}, 8},
      {4, 128, TWINKV_F32, {300, 129, 128, 127}, 8},
      {9, 64, TWINKV_BF16, {1000, 2048, 2049}, 0},
      {1, 128, TWINKV_BF16, {40000}, 0},
      {70, 128, TWINKV_BF16, {3, 2}, 0},
  };
  for (const Shape& sh : shapes) run_shape(sh);
  invalid_arguments();
  if (g_fail) {
    std::fprintf(stderr, "%d expectation(s) failed\n", g_fail);
    return 1;
  }
  std::printf("host layer ok: %lld stubbed launches\n", (long long)stub::g_launches);
  return 0;
}

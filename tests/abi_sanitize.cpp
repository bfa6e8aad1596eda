// Validation paths of the C ABI, run against a build of libifvs whose host
// code is compiled with AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_abi_sanitize.py builds both).  Every call below must return
// the documented status without touching the GPU: NULL handles and outputs,
// and every malformed index descriptor field.  A well-formed descriptor is
// then loaded: on a machine without a GPU the load fails with IFVS_E_HIP
// after the host has allocated and released its handle, with a GPU it
// succeeds and the handle is freed.  The process exits 0 when every status
// matched; any memory error or undefined behaviour aborts it.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "ifvs.h"

static int g_fail = 0;

static void expect(const char* what, ifvs_status got, ifvs_status want) {
  if (got != want) {
    std::fprintf(stderr, "FAIL %s: status %d, expected %d (%s)\n", what, got, want, ifvs_last_error());
    ++g_fail;
  }
}

int main() {
  const int64_t n = 1000;
  const int dim = 8, m = 4, dsub = dim / m;
  std::vector<uint8_t> codes(static_cast<size_t>(n) * m, 7);
  std::vector<float> codebook(static_cast<size_t>(m) * 256 * dsub, 0.5f);
  std::vector<int32_t> attrs(static_cast<size_t>(n), 3);
  std::vector<float> bank(static_cast<size_t>(16) * m * 2, 0.0f);
  std::vector<float> W(static_cast<size_t>(m) * 2 * 256 * dsub, 0.0f);

  ifvs_index_desc good;
  std::memset(&good, 0, sizeof(good));
  good.n = n;
  good.dim = dim;
  good.m = m;
  good.ksub = 256;
  good.n_attr = 1;
  good.codes = codes.data();
  good.codebook = codebook.data();
  good.attrs = attrs.data();
  good.bank_rows = 16;
  good.r = 2;
  good.h = 2;
  good.mem_kind = IFVS_MEM_HOST;
  good.hash_seed = 12345;
  good.bank = bank.data();
  good.W = W.data();
  good.max_batch = 8;
  good.max_k = 10;
  good.n_cluster = 1;
  good.cluster_col[0] = 0;

  // the error text is always a valid string
  if (!ifvs_last_error()) {
    std::fprintf(stderr, "FAIL ifvs_last_error returned NULL\n");
    ++g_fail;
  }

  // ---- ifvs_load_index: NULL arguments and every malformed field
  ifvs_index* idx = nullptr;
  expect("load NULL desc", ifvs_load_index(nullptr, &idx), IFVS_E_INVALID);
  expect("load NULL out", ifvs_load_index(&good, nullptr), IFVS_E_INVALID);
  struct Case {
    const char* what;
    void (*mutate)(ifvs_index_desc&);
  };
  const Case cases[] = {
      {"n = 0", [](ifvs_index_desc& d) { d.n = 0; }},
      {"n = 2^31", [](ifvs_index_desc& d) { d.n = int64_t(1) << 31; }},
      {"dim = 0", [](ifvs_index_desc& d) { d.dim = 0; }},
      {"dim = 5000", [](ifvs_index_desc& d) { d.dim = 5000; }},
      {"m = 0", [](ifvs_index_desc& d) { d.m = 0; }},
      {"m not dividing dim", [](ifvs_index_desc& d) { d.m = 3; }},
      {"m = 512", [](ifvs_index_desc& d) { d.m = 512; d.dim = 512; }},
      {"ksub = 16", [](ifvs_index_desc& d) { d.ksub = 16; }},
      {"n_attr = -1", [](ifvs_index_desc& d) { d.n_attr = -1; }},
      {"n_attr = 17", [](ifvs_index_desc& d) { d.n_attr = 17; }},
      {"mem_kind = 9", [](ifvs_index_desc& d) { d.mem_kind = 9; }},
      {"codes NULL", [](ifvs_index_desc& d) { d.codes = nullptr; }},
      {"codebook NULL", [](ifvs_index_desc& d) { d.codebook = nullptr; }},
      {"attrs NULL", [](ifvs_index_desc& d) { d.attrs = nullptr; }},
      {"bank_rows = -1", [](ifvs_index_desc& d) { d.bank_rows = -1; }},
      {"r = 0", [](ifvs_index_desc& d) { d.r = 0; }},
      {"r = 65", [](ifvs_index_desc& d) { d.r = 65; }},
      {"h = 0", [](ifvs_index_desc& d) { d.h = 0; }},
      {"h = 17", [](ifvs_index_desc& d) { d.h = 17; }},
      {"bank NULL", [](ifvs_index_desc& d) { d.bank = nullptr; }},
      {"W NULL", [](ifvs_index_desc& d) { d.W = nullptr; }},
      {"max_batch = 0", [](ifvs_index_desc& d) { d.max_batch = 0; }},
      {"max_batch = 65536", [](ifvs_index_desc& d) { d.max_batch = 65536; }},
      {"max_k = 0", [](ifvs_index_desc& d) { d.max_k = 0; }},
      {"max_k = 1025", [](ifvs_index_desc& d) { d.max_k = 1025; }},
      {"n_cluster = 3", [](ifvs_index_desc& d) { d.n_cluster = 3; }},
      {"n_cluster = -1", [](ifvs_index_desc& d) { d.n_cluster = -1; }},
      {"cluster_col = n_attr", [](ifvs_index_desc& d) { d.cluster_col[0] = 1; }},
      {"cluster_col = -1", [](ifvs_index_desc& d) { d.cluster_col[0] = -1; }},
      {"equal cluster columns", [](ifvs_index_desc& d) {
         d.n_cluster = 2;
         d.cluster_col[1] = 0;
       }},
  };
  for (const Case& c : cases) {
    ifvs_index_desc d = good;
    c.mutate(d);
    idx = reinterpret_cast<ifvs_index*>(0x1);
    expect(c.what, ifvs_load_index(&d, &idx), IFVS_E_INVALID);
    if (idx != nullptr) {
      std::fprintf(stderr, "FAIL %s: *out not cleared\n", c.what);
      ++g_fail;
    }
    if (std::strlen(ifvs_last_error()) == 0) {
      std::fprintf(stderr, "FAIL %s: empty error text\n", c.what);
      ++g_fail;
    }
  }

  // ---- every entry point on a NULL handle
  float f[64] = {};
  int32_t i32[64] = {};
  int64_t i64[128] = {};
  double dbl[16] = {};
  uint32_t u32[64] = {};
  uint8_t u8[64] = {};
  ifvs_predicate pred;
  std::memset(&pred, 0, sizeof(pred));
  expect("select_codebook", ifvs_select_codebook(nullptr, 1, f, &pred, nullptr, f, f, nullptr), IFVS_E_STATE);
  expect("build_lut", ifvs_build_lut(nullptr, 1, f, nullptr, f, 0, f, nullptr), IFVS_E_STATE);
  expect("build_sdc_lut", ifvs_build_sdc_lut(nullptr, 1, f, 0, f, nullptr), IFVS_E_STATE);
  expect("filter", ifvs_filter(nullptr, 1, &pred, u32, i64, nullptr), IFVS_E_STATE);
  expect("filtered_search", ifvs_filtered_search(nullptr, 1, &pred, f, 0, 1, i32, f, nullptr, nullptr),
         IFVS_E_STATE);
  expect("filtered_search_noalloc",
         ifvs_filtered_search_noalloc(nullptr, 1, &pred, f, 0, 1, i32, f, nullptr, nullptr), IFVS_E_STATE);
  expect("build_coarse", ifvs_build_coarse(nullptr, 16, 1), IFVS_E_STATE);
  expect("lut_bounds", ifvs_lut_bounds(nullptr, 1, nullptr, nullptr, f, nullptr), IFVS_E_STATE);
  expect("filtered_search_bounded",
         ifvs_filtered_search_bounded(nullptr, 1, &pred, f, 0, nullptr, nullptr, 1, i32, f, nullptr, nullptr),
         IFVS_E_STATE);
  expect("query_batch",
         ifvs_query_batch(nullptr, 1, f, &pred, f, nullptr, f, f, 0, f, 1, i32, f, nullptr), IFVS_E_STATE);
  expect("read_coarse", ifvs_read_coarse(nullptr, i32, nullptr, nullptr, u8), IFVS_E_STATE);
  expect("last_coarse", ifvs_last_coarse(nullptr, i32), IFVS_E_STATE);
  expect("load_vectors", ifvs_load_vectors(nullptr, f, IFVS_MEM_HOST), IFVS_E_STATE);
  expect("train_step",
         ifvs_train_step(nullptr, 1, f, &pred, f, i32, 1, 1, 1.0f, 0.0f, 0.1f, f, f, nullptr), IFVS_E_STATE);
  expect("read_params", ifvs_read_params(nullptr, f, f, nullptr), IFVS_E_STATE);
  expect("load_reconstructions", ifvs_load_reconstructions(nullptr), IFVS_E_STATE);
  expect("exact_search", ifvs_exact_search(nullptr, 1, f, &pred, 1, i32, f, nullptr), IFVS_E_STATE);
  expect("load_encoder", ifvs_load_encoder(nullptr, nullptr), IFVS_E_STATE);
  expect("encode_predicates", ifvs_encode_predicates(nullptr, 1, &pred, f, nullptr), IFVS_E_STATE);
  expect("set_option", ifvs_set_option(nullptr, IFVS_OPT_SPLITS, 1), IFVS_E_STATE);
  expect("read_profile", ifvs_read_profile(nullptr, dbl, i64), IFVS_E_STATE);
  expect("read_scan_reads", ifvs_read_scan_reads(nullptr, i64, nullptr), IFVS_E_STATE);
  expect("last_plan", ifvs_last_plan(nullptr, i64), IFVS_E_STATE);
  expect("probe active_lanes 0", ifvs_probe_lds_gather(0, dbl, nullptr), IFVS_E_INVALID);
  expect("probe NULL output", ifvs_probe_lds_gather(8, nullptr, nullptr), IFVS_E_INVALID);
  ifvs_free_index(nullptr);
  // the encoder's parameter count is host arithmetic: positive for a valid
  // shape, negative for an invalid one
  if (ifvs_encoder_params(64, 4, 2, 128, 1, dim) <= 0 || ifvs_encoder_params(0, 4, 2, 128, 1, dim) >= 0) {
    std::fprintf(stderr, "FAIL ifvs_encoder_params\n");
    ++g_fail;
  }

  // ---- a well-formed descriptor: loads with a GPU, IFVS_E_HIP without one
  idx = nullptr;
  const ifvs_status st = ifvs_load_index(&good, &idx);
  if (st == IFVS_OK) {
    ifvs_free_index(idx);
  } else if (st != IFVS_E_HIP || idx != nullptr) {
    std::fprintf(stderr, "FAIL well-formed load: status %d (%s)\n", st, ifvs_last_error());
    ++g_fail;
  }

  if (g_fail) return 1;
  std::printf("abi_sanitize: all statuses as documented\n");
  return 0;
}

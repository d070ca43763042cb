// Host-side checks of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer (test only; built and run by
// tests/test_host_sanitizers.py).  Exercises the pure host functions (shape
// checks, size queries, tree and mask validation, tree metadata) on valid,
// boundary and malformed inputs, and every call's argument checks with null
// or bad arguments, including context creation failing part way (no GPU, or
// the stubbed kernels) and the cleanup that follows.  Exit status 0 = every
// check held; the sanitizers abort on the first memory or UB error.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "tss.h"

static int failures = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static tss_model_cfg cfg7b() {
  tss_model_cfg c{};
  c.n_layers = 32; c.d_model = 4096; c.n_heads = 32; c.head_dim = 128; c.ffn_dim = 11008; c.vocab = 32000;
  c.rope_base = 10000.f; c.rms_eps = 1e-6f; c.dtype = TSS_BF16; c.max_nodes = 64; c.max_batch = 1;
  return c;
}

static void shapes() {
  tss_model_cfg c = cfg7b();
  CHECK(tss_cfg_check(&c) == TSS_OK);
  CHECK(tss_cfg_check(nullptr) == TSS_EINVAL);
  CHECK(tss_weights_bytes(nullptr) == 0 && tss_workspace_bytes(nullptr) == 0);
  CHECK(tss_kv_bytes(&c, 0, 16) == 0 && tss_kv_bytes(&c, 1, 0) == 0 && tss_kv_bytes(nullptr, 1, 16) == 0);
  CHECK(tss_kv_bytes(&c, 8, 4096) > tss_kv_bytes(&c, 1, 4096));
  CHECK(tss_sweep_prefix_bytes(&c, 0) == 0 && tss_sweep_prefix_bytes(&c, 65) == 0);
  CHECK(tss_sweep_prefix_bytes(&c, 33) == (size_t)32 * 33 * 4096 * 4);
  // every field out of range in turn
  struct Bad { int32_t* f; int32_t v; };
  for (int i = 0; i < 12; ++i) {
    tss_model_cfg b = cfg7b();
    const Bad bad[12] = {{&b.n_layers, 0},  {&b.n_layers, 257}, {&b.head_dim, 96},   {&b.d_model, 4000},
                         {&b.vocab, 32001}, {&b.ffn_dim, 11000}, {&b.max_nodes, 0},  {&b.max_nodes, 65},
                         {&b.max_batch, 0}, {&b.max_batch, 9},  {&b.dtype, 7},      {&b.n_heads, 31}};
    *bad[i].f = bad[i].v;
    CHECK(tss_cfg_check(&b) == TSS_EINVAL);
    CHECK(tss_weights_bytes(&b) == 0 && tss_workspace_bytes(&b) == 0);
  }
  tss_model_cfg b = cfg7b();
  b.rms_eps = 0.f;
  CHECK(tss_cfg_check(&b) == TSS_EINVAL);
  b = cfg7b();
  b.rope_base = -1.f;
  CHECK(tss_cfg_check(&b) == TSS_EINVAL);
}

static void trees() {
  int32_t chain[64], depth[64];
  uint64_t anc[64];
  for (int i = 0; i < 64; ++i) chain[i] = i - 1;
  CHECK(tss_validate_tree(chain, 64, 64) == TSS_OK);
  CHECK(tss_validate_tree(nullptr, 64, 64) == TSS_OK);
  CHECK(tss_validate_tree(chain, 65, 64) == TSS_EINVAL);
  CHECK(tss_validate_tree(chain, 64, 63) == TSS_EINVAL);
  CHECK(tss_validate_tree(chain, 0, 64) == TSS_EINVAL);
  CHECK(tss_validate_tree(chain, -5, 64) == TSS_EINVAL);
  int32_t bad[4] = {-1, 0, 2, 1};   // node 2 names itself
  CHECK(tss_validate_tree(bad, 4, 64) == TSS_EINVAL);
  bad[2] = 3;                       // a later node
  CHECK(tss_validate_tree(bad, 4, 64) == TSS_EINVAL);
  bad[0] = 0;                       // root with a parent
  bad[2] = 1;
  CHECK(tss_validate_tree(bad, 4, 64) == TSS_EINVAL);
  bad[0] = -1;
  bad[3] = -2;                      // negative parent
  CHECK(tss_validate_tree(bad, 4, 64) == TSS_EINVAL);
  CHECK(tss_tree_meta(chain, 64, depth, anc) == TSS_OK);
  CHECK(depth[63] == 63 && anc[63] == ~0ull && anc[0] == 1ull);
  CHECK(tss_tree_meta(chain, 64, nullptr, anc) == TSS_EINVAL && tss_tree_meta(chain, 64, depth, nullptr) == TSS_EINVAL);
  CHECK(tss_tree_meta(bad, 4, depth, anc) == TSS_EINVAL);
  // random trees against a brute-force walk to the root
  std::mt19937 rng(42);
  for (int t = 0; t < 200; ++t) {
    const int n = 1 + (int)(rng() % 64);
    std::vector<int32_t> par(n);
    par[0] = -1;
    for (int i = 1; i < n; ++i) par[i] = (int32_t)(rng() % i);
    CHECK(tss_validate_tree(par.data(), n, 64) == TSS_OK);
    CHECK(tss_tree_meta(par.data(), n, depth, anc) == TSS_OK);
    for (int i = 0; i < n; ++i) {
      int d = 0;
      uint64_t a = 1ull << i;
      for (int j = i; par[j] >= 0; j = par[j]) {
        ++d;
        a |= 1ull << par[j];
      }
      CHECK(depth[i] == d && anc[i] == a);
    }
  }
}

static void masks() {
  std::vector<uint8_t> m(256, 0);
  CHECK(tss_validate_mask(m.data(), 256) == TSS_OK);
  CHECK(tss_validate_mask(nullptr, 32) == TSS_OK);
  CHECK(tss_validate_mask(m.data(), 0) == TSS_EINVAL && tss_validate_mask(m.data(), 257) == TSS_EINVAL);
  m[31] = 1;
  CHECK(tss_validate_mask(m.data(), 32) == TSS_OK);
  m[31] = 2;
  CHECK(tss_validate_mask(m.data(), 32) == TSS_EINVAL);
  CHECK(tss_validate_mask(m.data(), 31) == TSS_OK);
}

static void null_context_calls() {
  int32_t a = 0, b = 0, tok[2] = {1, 2};
  float f[4];
  double ms;
  int64_t cnt;
  CHECK(tss_load_weights(nullptr, 0, 1, nullptr) == TSS_EINVAL);
  CHECK(tss_kv_alloc(nullptr, 1, 16, nullptr, 0, nullptr) == TSS_EINVAL);
  CHECK(tss_set_skip_mask(nullptr, 0, nullptr) == TSS_EINVAL);
  CHECK(tss_prefill(nullptr, 0, tok, 2) == TSS_EINVAL);
  CHECK(tss_verify(nullptr, 0, tok, nullptr, 2, nullptr, 0, &a, &b) == TSS_EINVAL);
  CHECK(tss_verify_batch(nullptr, 1, &a, &a, tok, nullptr, nullptr, 0, &a, &b) == TSS_EINVAL);
  CHECK(tss_verify_sweep(nullptr, 0, tok, nullptr, 2, 1, nullptr, &a, &b, nullptr, nullptr, 0) == TSS_EINVAL);
  CHECK(tss_get_logits(nullptr, f, 1) == TSS_EINVAL && tss_get_greedy(nullptr, &a, 1) == TSS_EINVAL);
  CHECK(tss_get_logits_device(nullptr, f, 1) == TSS_EINVAL);
  CHECK(tss_get_path(nullptr, 0, &a, &b) == TSS_EINVAL);
  CHECK(tss_get_attn_split(nullptr, &a, &a, &b) == TSS_EINVAL);
  CHECK(tss_check_kv(nullptr) == TSS_EINVAL);
  CHECK(tss_seq_length(nullptr, 0, &a) == TSS_EINVAL && tss_seq_truncate(nullptr, 0, 0) == TSS_EINVAL);
  CHECK(tss_set_launch_mode(nullptr, 0) == TSS_EINVAL);
  CHECK(tss_profile_kernel(nullptr, 0, 0) == TSS_EINVAL && tss_profile_read(nullptr, &ms, &cnt, 0) == TSS_EINVAL);
  CHECK(std::strlen(tss_last_error(nullptr)) > 0);
  for (int s = 1; s >= -6; --s) CHECK(std::strlen(tss_status_string(s)) > 0);
  tss_destroy(nullptr);
}

static void create_paths() {
  tss_model_cfg c = cfg7b();
  c.n_layers = 2;
  tss_ctx* ctx = reinterpret_cast<tss_ctx*>(0x1);
  uint8_t dummy[16];
  CHECK(tss_create(&c, nullptr, dummy, 16, dummy, 16, nullptr) == TSS_EINVAL);
  CHECK(tss_create(nullptr, nullptr, dummy, 16, dummy, 16, &ctx) == TSS_EINVAL && ctx == nullptr);
  CHECK(tss_create(&c, nullptr, nullptr, 16, dummy, 16, &ctx) == TSS_EINVAL && ctx == nullptr);
  CHECK(tss_create(&c, nullptr, dummy, 16, nullptr, 16, &ctx) == TSS_EINVAL && ctx == nullptr);
  CHECK(tss_create(&c, nullptr, dummy, 16, dummy, 16, &ctx) == TSS_ENOSPACE && ctx == nullptr);
  // full sizes: creation runs its HIP set-up, which fails without a GPU or at
  // the stubbed kernel attributes; the partly built context must be released
  const size_t wb = tss_weights_bytes(&c), sb = tss_workspace_bytes(&c);
  const int st = tss_create(&c, nullptr, dummy, wb, dummy, sb, &ctx);
  CHECK(st == TSS_EHIP && ctx == nullptr);
  CHECK(std::strstr(tss_last_error(nullptr), "tss_create") != nullptr);
}

int main() {
  shapes();
  trees();
  masks();
  null_context_calls();
  create_paths();
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("host sanitizer checks passed\n");
  return 0;
}

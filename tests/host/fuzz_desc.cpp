// fuzz_desc.cpp - seeded fuzzer of libfavor's host layer (argument validation,
// workspace sizing and launch planning), built for the CPU with address and
// undefined-behaviour sanitizers against stubs.cpp. For random descriptors,
// pointers and workspace sizes it checks that
//   * nothing crashes or overflows (the sanitizers abort on any finding);
//   * a call that returns an error launched nothing, and left a message;
//   * a workspace size is non-zero only for a descriptor that validates, and
//     a call with the size it reports gets past the workspace check;
//   * every launch the host layer makes has consistent arguments (stubs.cpp).
// Usage: fuzz_desc SEED ITERATIONS
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>

#include "../../include/favor.h"

extern int g_launches;

namespace {

uint64_t g_state;
uint64_t next() {   // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
template <typename T, size_t N>
T pick(const T (&a)[N]) { return a[next() % N]; }
bool coin(int pct) { return (int)(next() % 100) < pct; }

int fails = 0;
void check(bool ok, const char *what, long iter) {
  if (!ok) {
    std::fprintf(stderr, "iteration %ld: %s\n", iter, what);
    ++fails;
  }
}

favor_desc random_desc() {
  favor_desc g;
  std::memset(&g, 0, sizeof g);
  if (coin(15)) {   // raw garbage in every field
    uint32_t w[sizeof(favor_desc) / 4];
    for (auto &x : w) x = (uint32_t)next();
    std::memcpy(&g, w, sizeof g);
    return g;
  }
  const int32_t Bs[] = {0, 1, 2, 4, 8, -1, 255, 256, 65535, 65536, INT_MAX, INT_MIN};
  const int32_t Ls[] = {0, 1, 17, 63, 64, 65, 1000, 8192, 65536, 1 << 24, INT_MAX,
                        INT_MAX - 63, INT_MAX - 64, -1, INT_MIN};
  const int32_t ds[] = {64, 64, 64, 0, -64, 16, 32, 128, 65};
  const int32_t Ms[] = {16, 48, 64, 100, 128, 144, 240, 256, 0, 8, 272, 512, 4096, -16, INT_MAX};
  const int32_t dts[] = {0, 1, 0, 1, 2, -1};
  const float fs[] = {0.35355339f, 1.f, 0.f, -1.f, 1e30f, std::numeric_limits<float>::infinity(),
                      std::numeric_limits<float>::quiet_NaN()};
  const float eps[] = {0.f, 0.f, 1e-6f, 0.5f, -1e-3f, std::numeric_limits<float>::quiet_NaN(),
                       std::numeric_limits<float>::infinity()};
  const int32_t chunks[] = {0, 0, 64, 128, 192, 1024, 100, -64, INT_MAX, INT_MAX - 63, 1 << 30};
  const int32_t vT[] = {0, 64, 0, 64, 32, 128, -1};
  const int32_t kernels[] = {0, 1, 0, 2, -1};
  const int32_t rn[] = {0, 0, 1, 2, -1};
  if (coin(60)) {   // a valid descriptor, then at most one field mutated below
    const int32_t vL[] = {1, 17, 63, 64, 65, 1000, 8192, 65536, 1 << 20, 1 << 30};
    const int32_t vM[] = {16, 48, 64, 112, 128, 144, 240, 256};
    const int32_t vc[] = {0, 0, 64, 192, 1024, 1 << 30};
    g.B = 1 + (int)(next() % 4);
    g.H = 1 + (int)(next() % 8);
    if (coin(5)) { g.B = 255; g.H = 257; }
    g.L = pick(vL);
    g.d = 64;
    g.M = pick(vM);
    g.in_dtype = (favor_dtype)(next() % 2);
    g.out_dtype = coin(70) ? g.in_dtype : (favor_dtype)(next() % 2);
    g.input_scale = coin(80) ? 0.35355339f : 1.f;
    g.denom_eps = coin(70) ? 0.f : 0.25f;
    g.segment = pick(vc);
    g.chunk = coin(80) ? 0 : 64;
    g.kernel = (int)(next() % 2);
    g.no_renormalize = coin(80) ? 0 : 1;
    g.kernel_eps = 1e-3f;
    if (coin(50)) return g;
    switch (next() % 14) {
      case 0: g.B = pick(Bs); break;
      case 1: g.H = pick(Bs); break;
      case 2: g.L = pick(Ls); break;
      case 3: g.d = pick(ds); break;
      case 4: g.M = pick(Ms); break;
      case 5: g.in_dtype = (favor_dtype)pick(dts); break;
      case 6: g.out_dtype = (favor_dtype)pick(dts); break;
      case 7: g.input_scale = pick(fs); break;
      case 8: g.denom_eps = pick(eps); break;
      case 9: g.segment = pick(chunks); break;
      case 13: g.chunk = pick(vT); break;
      case 10: g.kernel = pick(kernels); break;
      default: g.no_renormalize = pick(rn); break;
    }
    return g;
  }
  g.B = coin(80) ? pick(Bs) % 9 : pick(Bs);
  g.H = coin(80) ? pick(Bs) % 9 : pick(Bs);
  if (g.B < 0 && g.B != INT_MIN && coin(50)) g.B = -g.B;
  g.L = pick(Ls);
  g.d = pick(ds);
  g.M = pick(Ms);
  g.in_dtype = (favor_dtype)pick(dts);
  g.out_dtype = (favor_dtype)pick(dts);
  g.input_scale = pick(fs);
  g.denom_eps = pick(eps);
  g.segment = pick(chunks);
  g.chunk = pick(vT);
  g.kernel = pick(kernels);
  g.no_renormalize = pick(rn);
  g.kernel_eps = pick(eps);
  return g;
}

// A fake device pointer: null, misaligned or aligned (never dereferenced).
void *ptr() {
  const int k = (int)(next() % 40);
  if (k == 0) return nullptr;
  if (k == 1) return reinterpret_cast<void *>(0x100001ull + 2 * (next() % 1000));
  return reinterpret_cast<void *>(0x10000000ull + 256 * (next() % 100000));
}

size_t ws_bytes(size_t need) {
  switch (next() % 12) {
    case 0: return 0;
    case 1: return need ? need - 1 : 0;
    case 2: return SIZE_MAX;
    default: return need + (next() % 4096);
  }
}

void *ws_ptr() {
  const int k = (int)(next() % 30);
  if (k == 0) return nullptr;
  if (k == 1) return reinterpret_cast<void *>(0x20000000ull + 16 * (1 + next() % 15));
  return reinterpret_cast<void *>(0x20000000ull + 256 * (next() % 100000));
}

// One call of an entry point: an error means no launch and a message, and a
// workspace of at least the reported size is never too small.
size_t g_need = 0, g_given = 0;
size_t ws_for(size_t need) {
  g_need = need;
  g_given = ws_bytes(need);
  return g_given;
}
void call(long iter, const char *name, int before, favor_status st) {
  if (st == FAVOR_ERR_WORKSPACE_TOO_SMALL && g_given >= g_need) {
    std::fprintf(stderr, "iteration %ld: %s rejected %zu bytes of workspace, reported %zu\n",
                 iter, name, g_given, g_need);
    ++fails;
  }
  g_need = g_given = 0;
  if (st != FAVOR_OK) {
    if (g_launches != before) {
      std::fprintf(stderr, "iteration %ld: %s failed (%d) after launching\n", iter, name, st);
      ++fails;
    }
    check(std::strlen(favor_last_error()) > 0, "error without a message", iter);
  }
  check(st >= FAVOR_OK && st <= FAVOR_ERR_DEVICE, "status out of range", iter);
  check(favor_status_string(st) != nullptr, "status string", iter);
}

}  // namespace

int main(int argc, char **argv) {
  g_state = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
  const long iters = argc > 2 ? std::atol(argv[2]) : 20000;
  long valid = 0, launched = 0;
  for (long it = 0; it < iters; ++it) {
    const favor_desc g = random_desc();
    // validation and sizes agree
    for (int op = -1; op <= 7; ++op) (void)favor_validate_desc(&g, op);
    const int size_ops[] = {0, 1, 2};
    const int val_ops[] = {1, 2, 3};
    for (int k = 0; k < 3; ++k) {
      const size_t n = favor_workspace_size(&g, size_ops[k]);
      const bool ok = favor_validate_desc(&g, val_ops[k]) == FAVOR_OK;
      check(n == 0 || ok, "workspace size for an invalid descriptor", it);
      valid += ok;
    }
    for (int c = 0; c < 3; ++c) {
      const size_t n = favor_backward_workspace_size(&g, c);
      check(n == 0 || favor_validate_desc(&g, 4 + c) == FAVOR_OK,
            "backward workspace size for an invalid descriptor", it);
    }
    (void)favor_workspace_size(nullptr, 0);
    (void)favor_validate_desc(nullptr, 1);

    const int before = g_launches;
    const size_t nb = favor_workspace_size(&g, 0), nc = favor_workspace_size(&g, 1),
                 nboth = favor_workspace_size(&g, 2);
    const size_t nbb = favor_backward_workspace_size(&g, 0),
                 nbc = favor_backward_workspace_size(&g, 1),
                 nbboth = favor_backward_workspace_size(&g, 2);
    const favor_desc *gp = coin(97) ? &g : nullptr;
    int b0 = g_launches;
    call(it, "feature_map", b0, favor_feature_map(gp, ptr(), (float *)ptr(), (float *)ptr(),
                                                  ptr(), nullptr));
    b0 = g_launches;
    if (coin(50))
      call(it, "attn_bidir", b0,
           favor_attn_bidir(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(), ptr(),
                            ws_ptr(), ws_for(nb), nullptr));
    else
      call(it, "attn_bidir_save", b0,
           favor_attn_bidir_save(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(), ptr(),
                                 coin(30) ? (float *)ptr() : nullptr, ws_ptr(), ws_for(nb),
                                 nullptr));
    b0 = g_launches;
    if (coin(50))
      call(it, "attn_causal", b0,
           favor_attn_causal(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(), ptr(),
                             coin(30) ? (float *)ptr() : nullptr,
                             coin(30) ? (float *)ptr() : nullptr, ws_ptr(), ws_for(nc), nullptr));
    else
      call(it, "attn_causal_save", b0,
           favor_attn_causal_save(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(), ptr(),
                                  coin(30) ? (float *)ptr() : nullptr,
                                  coin(30) ? (float *)ptr() : nullptr,
                                  coin(30) ? (float *)ptr() : nullptr, ws_ptr(), ws_for(nc),
                                  nullptr));
    b0 = g_launches;
    call(it, "attn_both", b0,
         favor_attn_both(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(), ptr(), ptr(),
                         coin(30) ? (float *)ptr() : nullptr, coin(30) ? (float *)ptr() : nullptr,
                         coin(30) ? (float *)ptr() : nullptr, coin(30) ? (float *)ptr() : nullptr,
                         ws_ptr(), ws_for(nboth), nullptr));
    b0 = g_launches;
    const bool saved = coin(40);
    call(it, "attn_bidir_backward", b0,
         favor_attn_bidir_backward(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(),
                                   ptr(), saved ? ptr() : nullptr,
                                   saved ? (float *)ptr() : nullptr,
                                   coin(30) ? ws_ptr() : nullptr, (int32_t)(next() % 5) - 1,
                                   ptr(), ptr(), ptr(), ws_ptr(), ws_for(nbb), nullptr));
    b0 = g_launches;
    call(it, "attn_causal_backward", b0,
         favor_attn_causal_backward(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(),
                                    coin(30) ? (float *)ptr() : nullptr, ptr(),
                                    saved ? ptr() : nullptr, saved ? (float *)ptr() : nullptr,
                                    coin(30) ? ws_ptr() : nullptr, (int32_t)(next() % 5) - 1,
                                    coin(30) ? (float *)ptr() : nullptr, ptr(), ptr(), ptr(),
                                    coin(30) ? (float *)ptr() : nullptr, ws_ptr(), ws_for(nbc),
                                    nullptr));
    b0 = g_launches;
    const bool saved_c = coin(40);
    call(it, "attn_both_backward", b0,
         favor_attn_both_backward(gp, ptr(), ptr(), ptr(), (float *)ptr(), (float *)ptr(),
                                  coin(30) ? (float *)ptr() : nullptr, ptr(), ptr(),
                                  saved ? ptr() : nullptr, saved ? (float *)ptr() : nullptr,
                                  saved_c ? ptr() : nullptr, saved_c ? (float *)ptr() : nullptr,
                                  coin(30) ? ws_ptr() : nullptr, (int32_t)(next() % 5) - 1,
                                  coin(30) ? (float *)ptr() : nullptr, ptr(), ptr(), ptr(),
                                  coin(30) ? (float *)ptr() : nullptr, ws_ptr(), ws_for(nbboth),
                                  nullptr));
    b0 = g_launches;
    const int32_t heads[] = {0, 1, 8, -1, 65535, 65536};
    const int32_t Ms[] = {64, 256, 100, 0, -1, 4096, 4097};
    const int32_t ds[] = {64, 32, 0};
    const int kinds[] = {0, 1, 2, 3, 4, 5, -1};
    call(it, "orf_draw", b0,
         favor_orf_draw(next(), pick(heads), pick(Ms), pick(ds), (favor_rf_kind)pick(kinds),
                        (float *)ptr(), (float *)ptr(), nullptr));
    launched += g_launches > before;
  }
  std::printf("fuzz: %ld iterations, %ld valid descriptor checks, %ld iterations launched, "
              "%d failures\n", iters, valid, launched, fails);
  return fails == 0 ? 0 : 1;
}

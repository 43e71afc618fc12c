// Host-side checks of the libwam C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (no GPU needed): size queries,
// configuration and argument validation, error strings, null handles, the
// allocation-free remap's and the probes' argument checks, and wam_init
// failing cleanly when no device can take the weights.  Exits non-zero on the
// first failed expectation; the sanitizers abort on any memory error or
// undefined behaviour.
#include <cstdio>
#include <cstring>
#include <vector>

#include "wam.h"

static int failures = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond);   \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

static wam_config cfg(int B, int L, int D, int H, int F, int Nv, int Cv, int Na, int A, int No, int Co, int dtype) {
  wam_config c{};
  c.B = B; c.L = L; c.D = D; c.H = H; c.F = F; c.Nv = Nv; c.Cv = Cv; c.Na = Na; c.A = A; c.No = No; c.Co = Co;
  c.dtype = dtype; c.qk_norm = 1; c.ln_eps = 1e-6f;
  return c;
}

int main() {
  // status strings
  for (int s = -6; s <= 0; ++s) EXPECT(std::strlen(wam_status_string(s)) > 0);
  EXPECT(std::strlen(wam_status_string(-99)) > 0);

  // size queries: the four workload shapes are valid, broken ones give 0
  const wam_config ok[] = {cfg(1, 2, 128, 4, 512, 64, 16, 16, 7, 8, 16, WAM_FP32),
                           cfg(1, 12, 768, 12, 3072, 768, 16, 32, 7, 64, 16, WAM_BF16),
                           cfg(4, 24, 1024, 16, 4096, 2000, 16, 50, 14, 256, 16, WAM_BF16),
                           cfg(1, 28, 1536, 24, 6144, 9600, 16, 64, 14, 512, 16, WAM_BF16)};
  for (const auto& c : ok) {
    EXPECT(wam_host_weight_count(&c) > 0);
    EXPECT(wam_weight_bytes(&c) > 0);
    EXPECT(wam_workspace_bytes(&c) > 0);
    EXPECT(wam_traj_elems(&c) == (int64_t)c.Nv * c.Cv + (int64_t)c.Na * c.A);
  }
  const wam_config bad[] = {cfg(0, 2, 128, 4, 512, 64, 16, 16, 7, 8, 16, WAM_FP32),    // no batch
                            cfg(17, 2, 128, 4, 512, 64, 16, 16, 7, 8, 16, WAM_FP32),   // batch > max
                            cfg(1, 2, 130, 4, 512, 64, 16, 16, 7, 8, 16, WAM_FP32),    // D % 64
                            cfg(1, 2, 128, 3, 512, 64, 16, 16, 7, 8, 16, WAM_FP32),    // D % H
                            cfg(1, 2, 128, 4, 512, 0, 16, 0, 7, 8, 16, WAM_FP32),      // no tokens
                            cfg(1, 2, 128, 4, 512, 64, 17, 16, 7, 8, 16, WAM_FP32),    // Cv > 16
                            cfg(1, 2, 128, 4, 512, 64, 16, 16, 7, 8, 16, 7)};          // dtype
  for (const auto& c : bad) {
    EXPECT(wam_host_weight_count(&c) == 0);
    EXPECT(wam_weight_bytes(&c) == 0);
    EXPECT(wam_workspace_bytes(&c) == 0);
  }
  EXPECT(wam_host_weight_count(nullptr) == 0);

  // wam_init argument checks (before any device work)
  wam_t h = nullptr;
  const wam_config& c0 = ok[0];
  const size_t nw = wam_host_weight_count(&c0);
  std::vector<float> w(nw, 0.01f);
  EXPECT(wam_init(nullptr, w.data(), nw, nullptr, 0, nullptr, 0, nullptr, &h) != WAM_OK);
  EXPECT(wam_init(&bad[2], w.data(), nw, nullptr, 0, nullptr, 0, nullptr, &h) != WAM_OK);
  EXPECT(wam_init(&c0, w.data(), nw - 1, nullptr, 0, nullptr, 0, nullptr, &h) != WAM_OK);
  EXPECT(wam_init(&c0, nullptr, nw, nullptr, 0, nullptr, 0, nullptr, &h) != WAM_OK);
  EXPECT(wam_init(&c0, w.data(), nw, nullptr, 0, nullptr, 0, nullptr, nullptr) != WAM_OK);
  // buffers too small
  EXPECT(wam_init(&c0, w.data(), nw, (void*)0x1000, 16, (void*)0x2000, 16, nullptr, &h) == WAM_E_WORKSPACE);
  EXPECT(h == nullptr);

  // null handles
  float dummy[4] = {0, 0, 0, 0};
  EXPECT(wam_velocity(nullptr, 0, dummy, dummy, dummy, nullptr, nullptr) == WAM_E_ARG);
  EXPECT(wam_denoise_step(nullptr, 0, dummy, dummy, nullptr, nullptr) == WAM_E_ARG);
  EXPECT(wam_continue(nullptr, 0, 1, dummy, dummy, nullptr, -1, nullptr, nullptr) == WAM_E_ARG);
  EXPECT(wam_adapt_state(nullptr, WAM_ADAPT_RESET_ALL, nullptr) == WAM_E_ARG);
  EXPECT(wam_set_schedule(nullptr, dummy, 1) == WAM_E_ARG);
  EXPECT(wam_set_option(nullptr, WAM_OPT_GRAPHS, 0) == WAM_E_ARG);
  EXPECT(wam_replan(nullptr, nullptr, nullptr) == WAM_E_ARG);
  EXPECT(wam_sync(nullptr) == WAM_E_ARG);
  EXPECT(std::strlen(wam_last_error(nullptr)) > 0);
  wam_destroy(nullptr);

  // allocation-free remap: argument and size checks with messages
  wam_remap_args ra{};
  EXPECT(wam_remap_noalloc(nullptr, &ra, nullptr) == WAM_E_ARG);
  EXPECT(std::strlen(wam_noalloc_last_error()) > 0);
  wam_config big = ok[0];
  big.B = 17;
  EXPECT(wam_remap_noalloc(&big, &ra, nullptr) == WAM_E_SHAPE);
  EXPECT(std::strstr(wam_noalloc_last_error(), "batch") != nullptr);
  EXPECT(wam_remap_noalloc(&c0, &ra, nullptr) == WAM_E_ARG);  // null buffers
  ra.x_bar = ra.x_r = ra.noise = dummy;
  ra.x_out = dummy + 1;
  ra.sigma_r = 0.f;
  EXPECT(wam_remap_noalloc(&c0, &ra, nullptr) == WAM_E_ARG);  // sigma_r <= 0
  ra.sigma_r = 0.5f;
  ra.shift_action = -1;
  EXPECT(wam_remap_noalloc(&c0, &ra, nullptr) == WAM_E_ARG);  // negative shift

  // probes
  double r1 = 0, r2 = 0;
  EXPECT(wam_probe_mfma_bf16(nullptr, 2, 1, 1, dummy, &r1, &r2) == WAM_E_ARG);
  EXPECT(wam_probe_mfma_bf16(nullptr, 0, 0, 1, dummy, &r1, &r2) == WAM_E_ARG);
  EXPECT(wam_probe_copy(nullptr, dummy, dummy + 1, 15, 1, &r1, &r2) == WAM_E_ARG);

  if (failures) {
    std::fprintf(stderr, "%d host check(s) failed\n", failures);
    return 1;
  }
  std::printf("host ABI checks passed\n");
  return 0;
}

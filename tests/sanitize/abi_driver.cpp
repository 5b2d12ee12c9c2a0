// Host-only driver for the sanitizer build of the library (AddressSanitizer +
// UndefinedBehaviorSanitizer on the host code): every call below must fail
// validation, or compute on the host only, before anything touches a device.
// Exits 0 when every status is the documented one.
#include <cstdio>
#include <cstdint>
#include <cmath>

#include "soap.h"

static int failures = 0;
#define EXPECT(call, want)                                                             \
  do {                                                                                 \
    int got_ = (call);                                                                 \
    if (got_ != (want)) {                                                              \
      std::printf("FAIL %s: got %d want %d (%s)\n", #call, got_, (int)(want),          \
                  soap_last_error());                                                  \
      ++failures;                                                                      \
    }                                                                                  \
  } while (0)

int main() {
  const uintptr_t base = 0x7f0000000000ull, mb = 1ull << 24;
  float *p[9];
  for (int i = 0; i < 9; ++i) p[i] = reinterpret_cast<float *>(base + i * mb);
  void *ws = p[8];
  // workspace sizes over many shapes and batches (layout arithmetic)
  size_t prev = 0;
  for (int64_t d = 1; d <= SOAP_MAX_DIM; d = d * 3 + 1) {
    for (int64_t b : {int64_t(1), int64_t(7), int64_t(64)}) {
      const size_t a = soap_workspace_bytes(b, d, d + 5), k = soap_kl_workspace_bytes(b, d, d + 5);
      const size_t off = soap_workspace_update_offset(b, d, d + 5);
      if (a == 0 || k < a || off + 4u * (size_t)b * d * (d + 5) > a || off % 256) {
        std::printf("FAIL layout b=%lld d=%lld: %zu %zu %zu\n", (long long)b, (long long)d, a, k, off);
        ++failures;
      }
    }
    const size_t q = soap_qr_workspace_bytes(d);
    if (q <= prev) { std::printf("FAIL qr workspace not increasing at %lld\n", (long long)d); ++failures; }
    prev = q;
    const int64_t e = 2 * d <= SOAP_MAX_DIM ? 2 * d : SOAP_MAX_DIM;
    if (soap_muon_workspace_bytes(1, d, e) == 0 || soap_kl_factors_workspace_bytes(d, d) == 0) {
      std::printf("FAIL muon/kl-factors workspace at %lld\n", (long long)d); ++failures;
    }
  }
  if (soap_workspace_bytes(1, 0, 4) != 0 || soap_workspace_bytes(1, 4, SOAP_MAX_DIM + 1) != 0 ||
      soap_workspace_update_offset(0, 4, 4) != 0 || soap_qr_workspace_bytes(-3) != 0) {
    std::printf("FAIL invalid shapes must give 0\n"); ++failures;
  }
  const size_t need = soap_workspace_bytes(1, 8, 12);
  // soap_step: every validation path
  EXPECT(soap_step(nullptr, p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_NULL);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 0, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_SHAPE);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, 1.f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, NAN, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 0, 0, ws, need, nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 64, ws, need, nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need - 1, nullptr), SOAP_ERR_WORKSPACE);
  EXPECT(soap_step(p[0], reinterpret_cast<float *>(base + mb + 4), p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_ALIGN);
  EXPECT(soap_step(p[0], p[0], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_ALIAS);
  EXPECT(soap_step_batched(0, p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, ws, need, nullptr), SOAP_ERR_SHAPE);
  EXPECT(soap_kl_step(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1.5f, 1e-8f, 1e-3f, .1f, 1, 0, ws, soap_kl_workspace_bytes(1, 8, 12), nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_kl_factors_f32(8, 12, p[1], p[2], p[3], p[4], p[5], .95f, 1e-8f, nullptr, nullptr, ws, 16, nullptr), SOAP_ERR_WORKSPACE);
  const float coeffs[6] = {1.5f, -.5f, 0.f, 1.5f, -.5f, 0.f};
  EXPECT(soap_muon_step(p[0], p[1], p[6], 8, 12, .9f, 1e-3f, .1f, 0.f, coeffs, 2, 0, ws, soap_muon_workspace_bytes(1, 8, 12), nullptr), SOAP_ERR_HPARAM);
  EXPECT(soap_muon_step(p[0], p[1], p[6], 10, 12, .9f, 1e-3f, .1f, 1e-7f, coeffs, 2, SOAP_MUON_BF16, ws, soap_muon_workspace_bytes(1, 10, 12), nullptr), SOAP_ERR_SHAPE);
  EXPECT(soap_qr_f32(64, p[0], p[1], nullptr, ws, 16, nullptr), SOAP_ERR_WORKSPACE);
  EXPECT(soap_qr_f32(64, p[0], p[0], nullptr, ws, soap_qr_workspace_bytes(64), nullptr), SOAP_ERR_ALIAS);
  EXPECT(soap_gemm_f32(0, 0, 4, 4, 4, 1.f, p[0], 2, p[1], 4, 0.f, p[2], 4, nullptr), SOAP_ERR_SHAPE);
  EXPECT(soap_factor_ema_f32(0, 4, 4, p[0], p[0], .5f, nullptr), SOAP_ERR_ALIAS);
  EXPECT(soap_init_state(1, 4, 4, reinterpret_cast<float *>(base + 8), nullptr, nullptr, nullptr, nullptr, nullptr, nullptr), SOAP_ERR_ALIGN);
  EXPECT(soap_step_noalloc(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], 4096, 4096, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, nullptr), SOAP_ERR_WORKSPACE);
  EXPECT(soap_step_noalloc(p[0], nullptr, p[2], p[3], p[4], p[5], p[6], p[7], 8, 12, .9f, .95f, 1e-8f, 1e-3f, .1f, 1, 0, nullptr), SOAP_ERR_NULL);
  EXPECT(soap_workspace_status(nullptr, nullptr, nullptr), SOAP_ERR_NULL);
  EXPECT(soap_test_force_qr_give_up(8), SOAP_ERR_HPARAM);
  EXPECT(soap_test_force_qr_give_up(0), SOAP_OK);
  // host-side measurement API
  for (int i = -1; i <= soap_timing_num_stages(); ++i) (void)soap_timing_stage_name(i);
  double ms = -1; int64_t n = -1; double fl = -1;
  EXPECT(soap_timing_reset(), SOAP_OK);
  EXPECT(soap_timing_get(0, &ms, &n, &fl), SOAP_OK);
  EXPECT(soap_timing_get(soap_timing_num_stages(), &ms, &n, &fl), SOAP_ERR_SHAPE);
  if (ms != 0.0 || n != 0 || fl != 0.0) { std::printf("FAIL timing totals not reset\n"); ++failures; }
  std::printf("%s (%d failures)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}

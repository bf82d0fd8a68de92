// Host-only stand-ins for the kernel launchers, linked with abi.cpp into a
// sanitizer build of the C ABI's argument checks.  The checks run before any
// launch, and the tests that use this build pass only arguments the checks
// reject, so reaching a stub is itself a failure: each one aborts.
#include <cstdio>
#include <cstdlib>

#include "../paper_2606_18114_amd/csrc/launchers.hpp"

namespace tmk {

[[noreturn]] static void reached(const char* name) {
  std::fprintf(stderr, "launcher %s reached in the host-only build\n", name);
  std::abort();
}

hipError_t launch_ternarize_pack(const float*, int64_t, int64_t, int, float, const float*,
                                 const float*, uint8_t*, float*, uint16_t*, uint64_t*,
                                 hipStream_t) {
  reached("ternarize_pack");
}
hipError_t launch_group_code_dot(const uint8_t*, const float*, int64_t, int64_t, int, float*,
                                 hipStream_t) {
  reached("group_code_dot");
}
hipError_t launch_scale_ste_grad(const float*, const uint8_t*, const float*, const float*,
                                 int64_t, int64_t, int, float, float*, float*, hipStream_t) {
  reached("scale_ste_grad");
}
hipError_t launch_tgemm_fwd(const uint16_t*, const uint8_t*, const float*, int64_t, int64_t,
                            int64_t, int, void*, bool, uint32_t*, hipStream_t) {
  reached("tgemm_fwd");
}
hipError_t launch_tgemm_bwd_dx(const uint16_t*, const uint8_t*, const float*, int64_t, int64_t,
                               int64_t, int, float*, hipStream_t) {
  reached("tgemm_bwd_dx");
}
hipError_t launch_tgemm_bwd_dx_f16(const uint16_t*, const uint8_t*, const float*, int64_t,
                                   int64_t, int64_t, int, float*, void*, hipStream_t) {
  reached("tgemm_bwd_dx_f16");
}
hipError_t launch_tgemm_bwd_dw(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t,
                               float*, int, hipStream_t) {
  reached("tgemm_bwd_dw");
}
hipError_t launch_fill_zero_f32(float*, int64_t, hipStream_t) { reached("fill_zero_f32"); }
bool tgemv_b16_takes(int B, int g) { return B >= 9 && B <= 16 && g >= 64 && g <= 512; }
hipError_t launch_tgemv_b16(const uint16_t*, const uint8_t*, const uint16_t*, int, int, int64_t,
                            int64_t, int, float*, hipStream_t) {
  reached("tgemv_b16");
}
hipError_t launch_tgemv(const uint16_t*, const uint8_t*, const uint16_t*, int, int, int64_t,
                        int64_t, int, float*, hipStream_t) {
  reached("tgemv");
}

hipError_t launch_tgemv_pair(const uint16_t*, const uint8_t*, const uint16_t*, int, int64_t,
                             int64_t, float*, const uint16_t*, const uint8_t*, const uint16_t*,
                             int, int64_t, int64_t, float*, int, int, hipStream_t) {
  reached("tgemv_pair");
}

hipError_t launch_dgemv(const uint16_t*, const uint16_t*, int, int, int64_t, int64_t, float*,
                        hipStream_t) {
  reached("dgemv");
}

hipError_t launch_tgemv_rms(const float*, const float*, float, const uint8_t*, const uint16_t*,
                            int, int64_t, int64_t, int, float*, int, hipStream_t) {
  reached("tgemv_rms");
}
hipError_t launch_dgemv_rms(const float*, const float*, float, const uint16_t*, int, int64_t,
                            int64_t, float*, int, hipStream_t) {
  reached("dgemv_rms");
}
hipError_t launch_mixer_gate(const float*, int, int, uint16_t*, int*, uint16_t*, const float*,
                             const float*, const float*, const float*, const float*, float*,
                             hipStream_t) {
  reached("mixer_gate");
}

hipError_t launch_mixer_step(const float*, int, int, uint16_t*, int*, uint16_t*, const float*,
                             const float*, const float*, const float*, const float*, const float*,
                             float, float*, uint16_t*, hipStream_t) {
  reached("mixer_step");
}

int64_t mixer_scratch_floats() { return 16 * (8192 + 128); }
hipError_t launch_mixer_step_noalloc(const float*, int, int, uint16_t*, int*, uint16_t*,
                                     const float*, const float*, const float*, const float*,
                                     const float*, const float*, float, uint16_t*, hipStream_t) {
  reached("mixer_step_noalloc");
}
hipError_t launch_decode_stack(const DecodeStackDesc&, const float*, uint16_t*, void*,
                               hipStream_t) {
  reached("decode_stack");
}
hipError_t launch_residual_rmsnorm(float*, const float*, int, int64_t, const float*, float,
                                   uint16_t*, hipStream_t) {
  reached("residual_rmsnorm");
}

}  // namespace tmk

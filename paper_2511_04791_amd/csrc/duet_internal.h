// Internal declarations shared by the host model, the runtime and the kernel launchers.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "duet.h"

namespace duet {

constexpr int kNumCuSteps = DUET_TOTAL_CUS / DUET_CU_STEP;  // 32 table entries: 8, 16, ..., 256

// Thread-local error message; every failing entry point sets it and returns the code.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Shape / batch checks shared by the model and the GPU path.
int check_shape(const duet_shape* s);
int check_batch(const duet_shape* s, const duet_batch* b, bool need_q_start);

}  // namespace duet

struct duet_model {
  double flops[duet::kNumCuSteps];  // Pi(S), FLOP/s, S = 8 (i + 1)
  double bytes[duet::kNumCuSteps];  // B(S), bytes/s
  // Rates of each share while the other half runs on the other CUs (spatial sharing); used
  // for the halves of a split batch holding both kinds when has_shared is set.
  double flops_shared[duet::kNumCuSteps];
  double bytes_shared[duet::kNumCuSteps];
  bool has_shared = false;
  // Fixed seconds per layer of each partition kind on S CUs, added once per layer when the batch
  // holds requests of that kind (kernel launches and the decode kernel's tail); zero by default,
  // which is the paper's model.
  double launch_prefill[duet::kNumCuSteps];
  double launch_decode[duet::kNumCuSteps];
  double prefill_eff = 1.0;
  double decode_eff = 1.0;
  bool calibrated = false;
};

namespace duet {
void model_init_nominal(duet_model* m);
}

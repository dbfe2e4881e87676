// host.h -- pieces shared by the host files of the library (dtr_sim.cpp for
// traces, dtr_log.cpp for operator logs): error reporting, heuristic and
// policy rules, bounds, and the log-replay plan.
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/dtr_sim.h"

namespace dtrhost {

constexpr int64_t MAX_SIZE = int64_t(1) << 36;
constexpr int64_t MAX_COST = int64_t(1) << 28;
constexpr int64_t MAX_TOTAL_COST = int64_t(1) << 50;
constexpr size_t ALIGN = 256;

int fail(int code, const char *fmt, ...);
bool heuristic_known(int32_t h);
// kernel specialisation: 0 union-find neighbourhood, 1 neighbourhood walk
// (e* or e_R), 2 no neighbourhood
int32_t heuristic_class(int32_t h);
// the spec rules shared by traces and logs (heuristic, policy, search flags)
int check_spec(const dtr_sim_spec &s, int32_t i);
int device_cus(int32_t *cus);
inline size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// operator-log replay (dtr_log.cpp)
struct LogPlan;
int log_plan_make(const dtr_log *logs, int32_t n_logs, const dtr_sim_spec *sims, int32_t n_sims,
                  const dtr_sim_options *opt, LogPlan **out);
size_t log_plan_total(const LogPlan *p);
size_t log_plan_result_off(const LogPlan *p);
int log_plan_upload(LogPlan *p, uint8_t *ws, hipStream_t st);
int log_plan_launch(const LogPlan *p, uint8_t *ws, hipStream_t st);
void log_plan_free(LogPlan *p);
// resident slots, waves per workgroup and dynamic LDS bytes of the launch
void log_plan_info(const LogPlan *p, int32_t *n_slots, int32_t *waves, int32_t *lds_bytes);

}  // namespace dtrhost

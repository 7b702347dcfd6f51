// Control-plane planners of the load-balancing orchestrator (Sec. 3.3): the
// resource partitioning plan (DP groups per policy version, in proportion to
// each version's workload) and the staleness-aware data supplementation
// (prompts for the latest version first, legacy versions only up to their
// idle slots).  Host code; integer arithmetic only.
#include <stdint.h>

#include <vector>

#include "dora.h"

extern "C" {

dora_status dora_plan_partition(const int64_t* workload, int32_t n_versions, int32_t n_groups,
                                int32_t* groups_out) {
  if (!workload || !groups_out || n_versions < 1 || n_groups < 1) return DORA_ERR_INVALID_ARG;
  int64_t total = 0;
  int32_t busy = 0;
  for (int32_t v = 0; v < n_versions; ++v) {
    if (workload[v] < 0) return DORA_ERR_INVALID_ARG;
    total += workload[v];
    busy += workload[v] > 0 ? 1 : 0;
  }
  if (busy > n_groups) return DORA_ERR_INVALID_ARG;  // every busy version needs a group
  for (int32_t v = 0; v < n_versions; ++v) groups_out[v] = 0;
  if (total == 0) {  // nothing to run: everything to the latest version
    groups_out[n_versions - 1] = n_groups;
    return DORA_OK;
  }
  // One group reserved for each version with work (no request is stranded);
  // the other R groups by the largest-remainder method on the quotas
  // R * workload / total, equal remainders going to the newer version (higher
  // index).
  const int64_t R = n_groups - busy;
  std::vector<int64_t> rem(n_versions, -1);
  int64_t given = 0;
  for (int32_t v = 0; v < n_versions; ++v) {
    if (workload[v] == 0) continue;
    const __int128 q = (__int128)workload[v] * R;  // quota numerator over `total`
    groups_out[v] = (int32_t)(1 + q / total);
    rem[v] = (int64_t)(q % total);
    given += groups_out[v];
  }
  for (; given < n_groups; ++given) {  // fewer than `busy` passes, one group each
    int32_t pick = -1;
    for (int32_t v = n_versions - 1; v >= 0; --v)
      if (rem[v] >= 0 && (pick < 0 || rem[v] > rem[pick])) pick = v;
    ++groups_out[pick];
    rem[pick] = -1;  // each version gains at most one remainder group
  }
  return DORA_OK;
}

dora_status dora_plan_supplement(const int32_t* groups, const int32_t* active,
                                 int32_t n_versions, int32_t slots_per_group,
                                 int64_t latest_quota, int32_t* inject_out) {
  if (!groups || !active || !inject_out || n_versions < 1 || slots_per_group < 1 ||
      latest_quota < 0)
    return DORA_ERR_INVALID_ARG;
  for (int32_t v = 0; v < n_versions; ++v)
    if (groups[v] < 0 || active[v] < 0) return DORA_ERR_INVALID_ARG;
  for (int32_t v = 0; v < n_versions; ++v) {
    const int64_t idle = (int64_t)groups[v] * slots_per_group - active[v];
    const int64_t free_slots = idle > 0 ? idle : 0;
    if (v == n_versions - 1)  // the latest version: up to the rollout batch still owed
      inject_out[v] = (int32_t)(free_slots < latest_quota ? free_slots : latest_quota);
    else  // legacy versions: only their residual idle slots
      inject_out[v] = (int32_t)free_slots;
  }
  return DORA_OK;
}

}  // extern "C"

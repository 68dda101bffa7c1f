// Error reporting and small helpers shared by the host sources of the library.
#pragma once
#include <string>

#include "adpsgd.h"
#include "schedule.hpp"

namespace adpsgd {

// Record msg as the calling thread's last error and return code.
int fail(int code, const std::string &msg);
// Clear the calling thread's last error; returns ADPSGD_OK.
int ok();

bool hparams_valid(const adpsgd_hparams *hp, std::string *why);
int32_t p_max_of(const adpsgd_hparams *hp);
// The schedule rules of hp, for period_at / sync_due / apply_sync.
SchedRule rule_of(const adpsgd_hparams *hp);

}  // namespace adpsgd

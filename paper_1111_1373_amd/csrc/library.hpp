// Internal interface between the translation units of libdtree (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <string>

#include "dtree.h"

namespace dtree {

// Message returned by dt_last_error() on the calling thread; returns `s`.
dt_status set_error(dt_status s, const std::string &msg);
dt_status set_hip_error(hipError_t e, const char *what);
void clear_error();

// Device and record width a tree or forest was created for.
int device_of(const dt_tree *t);
int device_of(const dt_forest *f);
int32_t features_of(const dt_tree *t);
int32_t features_of(const dt_forest *f);

}  // namespace dtree

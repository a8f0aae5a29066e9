// Host-side helpers that the library's C++ translation units share with
// model.hip: the per-thread error message behind sd_last_error() and the
// model's layer count.
#pragma once

#include <string>

#include "sd.h"

namespace sdk {

// Records msg as the calling thread's last error and returns st.
sd_status report(sd_status st, const std::string &msg);

// Layers of the model (0 for NULL).
int32_t model_layers(const sd_model *m);

}  // namespace sdk

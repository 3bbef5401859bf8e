// api.hpp -- helpers the C ABI's source files share: the calling thread's
// last-error text and the current device's compute-unit count.
#pragma once

#include "../../include/fgd.h"

namespace fgd {

// Records the printf-style message as the calling thread's last error
// (fgd_last_error) and returns st.
fgd_status api_fail(fgd_status st, const char *fmt, ...);

// Clears the calling thread's last error.
void api_clear();

// Compute units of the current device, queried once per device.
fgd_status api_device_cus(int &num_cus);

}  // namespace fgd

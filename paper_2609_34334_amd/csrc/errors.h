// The calling thread's error string, read by hoccl_last_error_string().
#pragma once

namespace hoccl {

void set_error_message(const char *msg);

}  // namespace hoccl

// Error reporting shared by the host-side sources of libsarathi.
#pragma once

namespace sarathi {

// Sets the calling thread's message (returned by sarathi_last_error) and
// returns `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

}  // namespace sarathi

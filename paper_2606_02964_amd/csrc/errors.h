// errors.h -- the thread-local message behind msa_last_error(), shared by
// every entry point of the library.
#pragma once

#include <string>

namespace msa {

void set_last_error(const std::string& msg);

}  // namespace msa

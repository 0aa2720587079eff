#pragma once

#include <string>
#include <vector>

namespace sobek {

// Prelude + plan source, as compiled.
std::string full_source(const std::string& plan_source);
// Content hash of the full source and compile options.
std::string jit_key(const std::string& plan_source);
// gfx950 code object for the plan source (from the disk cache when present).
// Throws std::runtime_error with the compiler log on failure.
std::vector<char> jit_compile(const std::string& plan_source, std::string* log = nullptr);

}  // namespace sobek

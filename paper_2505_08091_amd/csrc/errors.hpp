// Exception types that map onto the C ABI's status codes.
#pragma once

#include <stdexcept>
#include <string>

namespace lego {

struct Unsupported : std::logic_error {
  explicit Unsupported(const std::string& m) : std::logic_error(m) {}
};
struct HipFailure : std::runtime_error {
  explicit HipFailure(const std::string& m) : std::runtime_error(m) {}
};
struct NotBijective : std::logic_error {
  explicit NotBijective(const std::string& m) : std::logic_error(m) {}
};

}  // namespace lego

// Compile helper of the run-time specialisation: reads one specialised
// kernel source on stdin, compiles it with the runtime compiler this
// program is linked with (the ROCm installation's, whatever runtime the
// calling process has loaded), and writes to stdout a status byte (0 on
// success) followed by the code object, or by the compile log on failure.
#include <cstdio>
#include <iostream>
#include <iterator>
#include <string>
#include <vector>

namespace dg {
bool jit_compile_source(const std::string& src, std::vector<char>* code, std::string* log);
}

int main() {
  std::string src((std::istreambuf_iterator<char>(std::cin)), std::istreambuf_iterator<char>());
  std::vector<char> code;
  std::string log;
  const bool ok = !src.empty() && dg::jit_compile_source(src, &code, &log);
  const char status = ok ? 0 : 1;
  std::fwrite(&status, 1, 1, stdout);
  if (ok)
    std::fwrite(code.data(), 1, code.size(), stdout);
  else
    std::fwrite(log.data(), 1, log.size(), stdout);
  std::fflush(stdout);
  return ok ? 0 : 1;
}

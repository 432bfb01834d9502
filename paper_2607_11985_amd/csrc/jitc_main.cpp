// jitc_main.cpp -- vqc_jitc <kernel.hip> <code-object>: compiles one generated
// kernel (see jit_compile.cpp).  Touches no GPU.  Exit status 0 on success;
// the compiler's log goes to stderr.
#include <cstdio>
#include <fstream>
#include <iterator>
#include <string>
#include <vector>

#include "vqc.h"
#include "vqc_internal.h"

int main(int argc, char** argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: vqc_jitc <kernel.hip> <code-object>\n");
    return 2;
  }
  std::ifstream in(argv[1], std::ios::binary);
  if (!in) {
    std::fprintf(stderr, "vqc_jitc: cannot read %s\n", argv[1]);
    return 2;
  }
  const std::string src((std::istreambuf_iterator<char>(in)), std::istreambuf_iterator<char>());
  std::vector<char> code;
  std::string log;
  if (vqc::compile_source(src, code, log) != VQC_OK) {
    std::fprintf(stderr, "%s\n", log.c_str());
    return 1;
  }
  const std::string tmp = std::string(argv[2]) + ".part";
  FILE* f = std::fopen(tmp.c_str(), "wb");
  if (!f || std::fwrite(code.data(), 1, code.size(), f) != code.size() || std::fclose(f) != 0) {
    std::fprintf(stderr, "vqc_jitc: cannot write %s\n", argv[2]);
    return 2;
  }
  return std::rename(tmp.c_str(), argv[2]) == 0 ? 0 : 2;
}

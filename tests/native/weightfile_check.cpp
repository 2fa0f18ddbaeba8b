// Test driver for the host-only weight-file reader, built by the CPU tests
// with the address and undefined-behaviour sanitizers.
//
//   weightfile_check one FILE...    parse each file; print "status F F_logical"
//   weightfile_check prefixes FILE  parse every strict prefix of FILE; print
//                                   "length status" for each prefix that did
//                                   not fail with PAINN_E_FORMAT
//   weightfile_check flips FILE N   parse FILE with each of its first N bytes
//                                   replaced by 0x00, 0xff and 0x80 in turn;
//                                   print the count per status
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <fstream>
#include <iterator>
#include <map>
#include <string>
#include <vector>

#include "weightfile.h"

static std::vector<unsigned char> slurp(const char* path) {
  std::ifstream f(path, std::ios::binary);
  return std::vector<unsigned char>((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
}

// Parse from an exactly sized heap copy, so a read past the end is a
// sanitizer error rather than a read of the caller's larger buffer.
static int parse_exact(const std::vector<unsigned char>& src, size_t n, WeightFile* wf, std::string* err) {
  unsigned char* p = (unsigned char*)malloc(n ? n : 1);
  if (n) memcpy(p, src.data(), n);
  const int st = parse_weight_file(p, n, wf, err);
  free(p);
  return st;
}

int main(int argc, char** argv) {
  if (argc < 3) return 2;
  const std::string mode = argv[1];
  if (mode == "one") {
    for (int i = 2; i < argc; ++i) {
      std::vector<unsigned char> b = slurp(argv[i]);
      WeightFile wf;
      std::string err;
      const int st = parse_exact(b, b.size(), &wf, &err);
      printf("%d %d %d %s\n", st, st == PAINN_OK ? wf.hp.F : 0, st == PAINN_OK ? wf.hp.F_logical : 0,
             st == PAINN_OK ? "ok" : err.c_str());
    }
    return 0;
  }
  std::vector<unsigned char> b = slurp(argv[2]);
  if (mode == "prefixes") {
    for (size_t n = 0; n < b.size(); ++n) {
      WeightFile wf;
      std::string err;
      const int st = parse_exact(b, n, &wf, &err);
      if (st != PAINN_E_FORMAT) printf("%zu %d\n", n, st);
    }
    return 0;
  }
  if (mode == "flips" && argc >= 4) {
    const size_t nb = strtoul(argv[3], nullptr, 10);
    std::map<int, long> count;
    const unsigned char vals[3] = {0x00, 0xff, 0x80};
    for (size_t i = 0; i < nb && i < b.size(); ++i)
      for (unsigned char v : vals) {
        std::vector<unsigned char> c = b;
        c[i] = v;
        WeightFile wf;
        std::string err;
        ++count[parse_exact(c, c.size(), &wf, &err)];
      }
    for (auto& kv : count) printf("%d %ld\n", kv.first, kv.second);
    return 0;
  }
  return 2;
}

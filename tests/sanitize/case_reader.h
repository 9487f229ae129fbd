// Reader of the sanitizer drivers' case files (test infrastructure).
//
// Line format (one item per line, byte strings in hex, "-" for empty):
//   G <grammar file>        D <drop labels or ->        E <eos id>
//   V <n>  then n lines of hex spellings                S <n> <ids...>
//   L <n>  then per category "<name> <k>" and k lines of words
//   P <n>  then n lines of hex prefixes                 M <n> (masks to take)
#pragma once
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

struct Case {
  std::string grammar, drop;
  std::vector<std::string> vocab, prefixes;
  std::vector<int32_t> specials;
  int32_t eos = -1;
  std::vector<std::string> cat_names, cat_words;  // words '\n'-joined
  int n_masks = 0;
};

inline std::string unhex(const std::string& h) {
  if (h == "-") return std::string();
  std::string out;
  for (size_t i = 0; i + 1 < h.size(); i += 2) out.push_back((char)std::strtol(h.substr(i, 2).c_str(), nullptr, 16));
  return out;
}

inline std::string slurp(const std::string& path) {
  std::ifstream f(path, std::ios::binary);
  std::stringstream ss;
  ss << f.rdbuf();
  return ss.str();
}

inline bool read_case(const char* path, Case& c) {
  std::ifstream f(path);
  if (!f) return false;
  std::string tag;
  while (f >> tag) {
    if (tag == "G") {
      std::string p;
      f >> p;
      c.grammar = slurp(p);
    } else if (tag == "D") {
      f >> c.drop;
      if (c.drop == "-") c.drop.clear();
    } else if (tag == "E") {
      f >> c.eos;
    } else if (tag == "V" || tag == "P") {
      size_t n;
      f >> n;
      auto& dst = tag == "V" ? c.vocab : c.prefixes;
      for (size_t i = 0; i < n; ++i) {
        std::string h;
        f >> h;
        dst.push_back(unhex(h));
      }
    } else if (tag == "S") {
      size_t n;
      f >> n;
      for (size_t i = 0; i < n; ++i) {
        int32_t x;
        f >> x;
        c.specials.push_back(x);
      }
    } else if (tag == "L") {
      size_t n;
      f >> n;
      for (size_t i = 0; i < n; ++i) {
        std::string name;
        size_t k;
        f >> name >> k;
        std::string words;
        for (size_t j = 0; j < k; ++j) {
          std::string w;
          f >> w;
          if (j) words += '\n';
          words += w;
        }
        c.cat_names.push_back(name);
        c.cat_words.push_back(words);
      }
    } else if (tag == "M") {
      f >> c.n_masks;
    } else {
      std::fprintf(stderr, "unknown tag %s\n", tag.c_str());
      return false;
    }
  }
  return true;
}

inline void flatten(const std::vector<std::string>& v, std::vector<uint8_t>& bytes, std::vector<uint64_t>& off) {
  off.assign(1, 0);
  for (const auto& s : v) {
    bytes.insert(bytes.end(), s.begin(), s.end());
    off.push_back(bytes.size());
  }
  bytes.push_back(0);
}

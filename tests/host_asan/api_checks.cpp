// Host-side checks of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer: argument validation and workspace sizing of
// sa_api.hip, linked against launcher stand-ins that only count calls.
//
// Reads one case per line on stdin:
//   call <name> <expected rc> <needle in hex, "-" for none> <args...>
//   ws <call> <B> <H> <L_v> <L_a> <d> <block>
// Arguments are integers (pointers as addresses, NULL as 0) or floats, in
// the order of the C signature.  For a "call" case it checks the return
// code, that sa_last_error() holds the needle, and that a rejected call
// reached no launcher; for "ws" it prints the size.  Exit status 0 iff every
// case passed (a sanitizer report aborts the process).
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "sa.h"

extern "C" int sa_host_stub_launches;

namespace {

std::vector<std::string> tok;

void* P(size_t i) { return reinterpret_cast<void*>(static_cast<uintptr_t>(std::strtoull(tok[i].c_str(), nullptr, 0))); }
template <class T> T* Pt(size_t i) { return static_cast<T*>(P(i)); }
int I(size_t i) { return static_cast<int>(std::strtoll(tok[i].c_str(), nullptr, 0)); }
float F(size_t i) { return std::strtof(tok[i].c_str(), nullptr); }
size_t Z(size_t i) { return static_cast<size_t>(std::strtoull(tok[i].c_str(), nullptr, 0)); }

std::string unhex(const std::string& h) {
  if (h == "-") return "";
  std::string out;
  for (size_t i = 0; i + 1 < h.size(); i += 2) out += static_cast<char>(std::stoi(h.substr(i, 2), nullptr, 16));
  return out;
}

// Calls entry point `name` with the arguments starting at token a.
bool dispatch(const std::string& name, size_t a, int* rc) {
  const size_t n = tok.size() - a;
  auto need = [&](size_t k) {
    if (n != k) {
      std::printf("BAD %s: %zu arguments, expected %zu\n", name.c_str(), n, k);
      std::exit(2);
    }
  };
  if (name == "sa_sparse_attention") {
    need(17);
    *rc = sa_sparse_attention(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<float>(a + 4), I(a + 5),
                              I(a + 6), I(a + 7), I(a + 8), I(a + 9), F(a + 10), I(a + 11),
                              Pt<const int32_t>(a + 12), Pt<const int32_t>(a + 13), P(a + 14),
                              Z(a + 15), P(a + 16));
  } else if (name == "sa_sparse_attention_noalloc") {
    need(15);
    *rc = sa_sparse_attention_noalloc(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<float>(a + 4),
                                      I(a + 5), I(a + 6), I(a + 7), I(a + 8), I(a + 9),
                                      F(a + 10), I(a + 11), Pt<const int32_t>(a + 12),
                                      Pt<const int32_t>(a + 13), P(a + 14));
  } else if (name == "sa_build_block_mask") {
    need(18);
    *rc = sa_build_block_mask(P(a), P(a + 1), I(a + 2), I(a + 3), I(a + 4), I(a + 5), I(a + 6),
                              F(a + 7), I(a + 8), I(a + 9), Pt<const uint8_t>(a + 10),
                              Pt<int32_t>(a + 11), Pt<int32_t>(a + 12), Pt<uint8_t>(a + 13),
                              Pt<float>(a + 14), P(a + 15), Z(a + 16), P(a + 17));
  } else if (name == "sa_cross_scores") {
    need(19);
    *rc = sa_cross_scores(P(a), P(a + 1), P(a + 2), P(a + 3), I(a + 4), I(a + 5), I(a + 6),
                          I(a + 7), I(a + 8), I(a + 9), F(a + 10), I(a + 11), Pt<float>(a + 12),
                          Pt<float>(a + 13), Pt<float>(a + 14), I(a + 15), P(a + 16), Z(a + 17),
                          P(a + 18));
  } else if (name == "sa_cross_attention") {
    need(15);
    *rc = sa_cross_attention(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<float>(a + 4), I(a + 5),
                             I(a + 6), I(a + 7), I(a + 8), I(a + 9), I(a + 10), F(a + 11),
                             P(a + 12), Z(a + 13), P(a + 14));
  } else if (name == "sa_cross_scores_from_lse") {
    need(21);
    *rc = sa_cross_scores_from_lse(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<const float>(a + 4),
                                   Pt<const float>(a + 5), I(a + 6), I(a + 7), I(a + 8),
                                   I(a + 9), I(a + 10), I(a + 11), F(a + 12), I(a + 13),
                                   Pt<float>(a + 14), Pt<float>(a + 15), Pt<float>(a + 16),
                                   I(a + 17), P(a + 18), Z(a + 19), P(a + 20));
  } else if (name == "sa_cross_scores_pooled") {
    need(23);
    *rc = sa_cross_scores_pooled(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<const float>(a + 4),
                                 Pt<const float>(a + 5), I(a + 6), I(a + 7), I(a + 8),
                                 I(a + 9), I(a + 10), I(a + 11), F(a + 12), I(a + 13),
                                 Pt<float>(a + 14), Pt<float>(a + 15), Pt<float>(a + 16),
                                 I(a + 17), Pt<double>(a + 18), Pt<double>(a + 19), P(a + 20),
                                 Z(a + 21), P(a + 22));
  } else if (name == "sa_build_block_mask_pooled") {
    need(15);
    *rc = sa_build_block_mask_pooled(Pt<const double>(a), Pt<const double>(a + 1), I(a + 2),
                                     I(a + 3), I(a + 4), I(a + 5), F(a + 6), I(a + 7),
                                     I(a + 8), Pt<const uint8_t>(a + 9), Pt<int32_t>(a + 10),
                                     Pt<int32_t>(a + 11), Pt<uint8_t>(a + 12),
                                     Pt<float>(a + 13), P(a + 14));
  } else if (name == "sa_select_protected") {
    need(7);
    *rc = sa_select_protected(Pt<const float>(a), I(a + 1), I(a + 2), I(a + 3),
                              Pt<int32_t>(a + 4), Pt<uint8_t>(a + 5), P(a + 6));
  } else if (name == "sa_saliency_ema") {
    need(5);
    *rc = sa_saliency_ema(Pt<float>(a), Pt<const float>(a + 1), Z(a + 2), F(a + 3), P(a + 4));
  } else if (name == "sa_select_protected_tokens") {
    need(7);
    *rc = sa_select_protected_tokens(Pt<const float>(a), I(a + 1), I(a + 2), I(a + 3),
                                     Pt<int32_t>(a + 4), Pt<uint8_t>(a + 5), P(a + 6));
  } else if (name == "sa_protected_token_attention") {
    need(16);
    *rc = sa_protected_token_attention(P(a), P(a + 1), P(a + 2), P(a + 3), Pt<float>(a + 4),
                                       I(a + 5), I(a + 6), I(a + 7), I(a + 8), I(a + 9),
                                       F(a + 10), Pt<const int32_t>(a + 11), I(a + 12),
                                       P(a + 13), Z(a + 14), P(a + 15));
  } else if (name == "sa_cache_indicator") {
    need(20);
    *rc = sa_cache_indicator(P(a), P(a + 1), Pt<const uint8_t>(a + 2), P(a + 3), P(a + 4),
                             Pt<const float>(a + 5), Pt<const float>(a + 6), I(a + 7), I(a + 8),
                             I(a + 9), I(a + 10), I(a + 11), F(a + 12), F(a + 13), F(a + 14),
                             F(a + 15), Pt<float>(a + 16), P(a + 17), Z(a + 18), P(a + 19));
  } else {
    return false;
  }
  return true;
}

}  // namespace

int main() {
  std::string line;
  int cases = 0, failed = 0;
  while (std::getline(std::cin, line)) {
    std::istringstream is(line);
    tok.clear();
    for (std::string t; is >> t;) tok.push_back(t);
    if (tok.empty()) continue;
    if (tok[0] == "ws" && tok.size() == 8) {
      std::printf("ws %zu\n", sa_workspace_size(I(1), I(2), I(3), I(4), I(5), I(6), I(7)));
      continue;
    }
    if (tok[0] != "call" || tok.size() < 4) {
      std::printf("BAD line: %s\n", line.c_str());
      return 2;
    }
    ++cases;
    const int want = I(2);
    const std::string needle = unhex(tok[3]);
    const int before = sa_host_stub_launches;
    int rc = -1;
    if (!dispatch(tok[1], 4, &rc)) {
      std::printf("BAD call name %s\n", tok[1].c_str());
      return 2;
    }
    const std::string msg = sa_last_error();
    const bool launched = sa_host_stub_launches != before;
    const bool ok = rc == want && msg.find(needle) != std::string::npos &&
                    (rc == SA_OK || !launched);
    if (!ok) {
      ++failed;
      std::printf("FAIL %s: rc %d (want %d), launched %d, message \"%s\" (want \"%s\")\n",
                  tok[1].c_str(), rc, want, static_cast<int>(launched), msg.c_str(),
                  needle.c_str());
    }
  }
  std::printf("cases %d failed %d\n", cases, failed);
  return failed == 0 ? 0 : 1;
}

// Internal declarations shared by the libckpt sources.
#pragma once

#include <cstdint>
#include <exception>
#include <string>
#include <vector>

#include "../../include/ckpt.h"

namespace ckpt {

inline uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

// An error carried to the C boundary as (code, message).
struct Error : std::exception {
  int code;
  std::string msg;
  Error(int c, std::string m) : code(c), msg(std::move(m)) {}
  const char *what() const noexcept override { return msg.c_str(); }
};

[[noreturn]] inline void fail(int code, const std::string &msg) { throw Error(code, msg); }

// the thread-local message ckpt_last_error() returns
void set_last_error(const std::string &msg);

// ---------------------------------------------------------------- plans --
struct Plan {
  int32_t mode = CKPT_NONE;
  int32_t n = 0;
  bool keep_last = false;
  int32_t fanout = 0;          // RECURSIVE: k stored splits per level; 0 otherwise
  std::vector<int32_t> cuts;   // ascending; cut c keeps x_{c+1}
  uint64_t x = 0, y = 0, extra = 0;

  // half-open segments [lo, hi) of a one-level plan
  std::vector<std::pair<int32_t, int32_t>> segments() const {
    std::vector<std::pair<int32_t, int32_t>> s;
    int32_t lo = 0;
    for (int32_t c : cuts) {
      s.emplace_back(lo, c + 1);
      lo = c + 1;
    }
    s.emplace_back(lo, n);
    return s;
  }
};

struct Accounting {
  uint64_t ckpt = 0, arena = 0, grad = 0;
  uint64_t peak() const { return ckpt + arena + grad; }
};

Plan make_plan(int32_t n, const uint64_t *layer_bytes, const uint64_t *cut_bytes, uint64_t budget,
               int32_t mode, const int32_t *user_cuts, int32_t n_user_cuts, int32_t flags);
std::vector<uint8_t> serialize(const Plan &p);
// b: n+1 entries, a and q: n entries; slot = gradient slot bytes (0: the
// largest boundary), extra = fixed gradient buffers
Accounting account(const Plan &p, const std::vector<uint64_t> &b, const std::vector<uint64_t> &a,
                   const std::vector<uint64_t> &q, uint64_t slot = 0, uint64_t extra = 0);
uint64_t recursive_extra(int32_t n, int32_t k);
// Section 4.4's split of [lo, hi) for fan-out k: the boundaries
// lo + floor(j (hi - lo) / (k+1)), j = 1..k, strictly inside, ascending,
// without repeats.
std::vector<int32_t> rec_splits(int32_t lo, int32_t hi, int32_t k);
// Appendix A's budget search: the candidate budgets (ascending) and the GREEDY
// plan of the candidate with the lowest exact peak (ties: smaller budget).
std::vector<uint64_t> search_candidates(int32_t n, const uint64_t *lb, const uint64_t *cb);
Plan search_plan(int32_t n, const uint64_t *lb, const uint64_t *cb, const std::vector<uint64_t> &b,
                 const std::vector<uint64_t> &a, const std::vector<uint64_t> &q, uint64_t slot,
                 uint64_t extra, int32_t flags, uint64_t *budget, uint64_t *peak);

// ------------------------------------------------------ gradient graphs --
struct GraphNode {
  int32_t kind, of;              // CKPT_GNODE_*, the forward node it derives from
  std::vector<int32_t> inputs;   // node ids it reads
  uint64_t bytes;                // output bytes
  bool inplace;
};
struct GraphPlan {
  std::vector<GraphNode> nodes;
  int32_t n_forward = 0;         // forward nodes (ids 0 .. n_forward-1)
  std::vector<int32_t> flags;    // their CKPT_NODE_* flags
  std::vector<int32_t> order;    // execution order
  std::vector<int32_t> tag_of;   // node id -> memory block (-1: none)
  std::vector<uint64_t> tag_bytes;
  uint64_t peak = 0;
  int32_t n_mirror = 0;
};
// Alg. 2 and the section-3 allocator (graph.cpp)
GraphPlan make_graph_plan(int32_t n, const int32_t *pred_ptr, const int32_t *pred_idx,
                          const uint64_t *out_bytes, const int32_t *flags, const int32_t *mirror,
                          int32_t strategy);

}  // namespace ckpt

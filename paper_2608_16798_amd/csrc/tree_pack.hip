// Prefix-tree packing of a rollout's model calls (ClawGym II, Sec. 3.2.1; the trainable-token
// rule of Sec. 3.2.3).  Host code only: it turns the captured (context, response) token lists of
// each rollout into the packed positions, parent pointers and training rows that the GPU entry
// points consume.
//
// Tree per rollout: node 0 is the empty root; node 1 holds the first call's context (the task
// prompt, harness content).  A call attaches to the node whose accumulated history is the
// longest prefix of its context, found by a depth-first walk that only follows children whose
// content matches the context at the current offset (a node's history is a prefix of the
// context exactly when every node on its path matches).  The new node holds the context's
// remainder (not trainable) followed by the response (trainable) unless an identical sibling
// exists.  Packing is depth-first pre-order with an explicit stack.
#include <string.h>

#include <vector>

#include "rlk_internal.h"

namespace rlk {
namespace {

struct Node {
  int64_t hist_len = 0;
  std::vector<int32_t> content;
  std::vector<uint8_t> mask;
  std::vector<int> children;
};

// The deepest node whose history is a prefix of x[0, nx); ties go to the earliest node.
int attach_point(const std::vector<Node>& nodes, const int32_t* x, int64_t nx) {
  int best = 0;
  int64_t best_len = 0;
  std::vector<int> stack{0};
  while (!stack.empty()) {
    const int k = stack.back();
    stack.pop_back();
    const Node& n = nodes[k];
    if (n.hist_len > best_len || (n.hist_len == best_len && k < best)) {
      best = k;
      best_len = n.hist_len;
    }
    for (int c : n.children) {
      const Node& ch = nodes[c];
      const int64_t len = (int64_t)ch.content.size();
      if (n.hist_len + len <= nx && memcmp(ch.content.data(), x + n.hist_len, (size_t)len * sizeof(int32_t)) == 0)
        stack.push_back(c);
    }
  }
  return best;
}

void build_tree(const rlk_calls_t* c, int r, std::vector<Node>& nodes) {
  nodes.assign(1, Node());
  const int64_t c0 = c->call_off[r], c1 = c->call_off[r + 1];
  if (c1 > c0) {
    const int64_t nx = c->x_off[c0 + 1] - c->x_off[c0];
    if (nx > 0) {
      Node p;
      p.hist_len = nx;
      p.content.assign(c->x_tok + c->x_off[c0], c->x_tok + c->x_off[c0] + nx);
      p.mask.assign((size_t)nx, 0);
      nodes.push_back(std::move(p));
      nodes[0].children.push_back(1);
    }
  }
  std::vector<int32_t> content;
  std::vector<uint8_t> mask;
  for (int64_t k = c0; k < c1; ++k) {
    const int32_t* x = c->x_tok + c->x_off[k];
    const int64_t nx = c->x_off[k + 1] - c->x_off[k];
    const int32_t* y = c->y_tok + c->y_off[k];
    const int64_t ny = c->y_off[k + 1] - c->y_off[k];
    const int at = attach_point(nodes, x, nx);
    const int64_t h = nodes[at].hist_len;
    content.assign(x + h, x + nx);
    content.insert(content.end(), y, y + ny);
    mask.assign((size_t)(nx - h), 0);
    mask.insert(mask.end(), (size_t)ny, 1);
    if (content.empty()) continue;
    bool same = false;
    for (int ch : nodes[at].children)
      if (nodes[ch].content == content && nodes[ch].mask == mask) {
        same = true;
        break;
      }
    if (same) continue;
    Node n;
    n.hist_len = nx + ny;
    n.content = content;
    n.mask = mask;
    nodes.push_back(std::move(n));
    nodes[at].children.push_back((int)nodes.size() - 1);
  }
}

// Positions and rows of one rollout's tree (appended when the output arrays are given).
void pack_tree(const std::vector<Node>& nodes, rlk_tree_out_t* o, bool write, int64_t& npos, int64_t& nrows) {
  struct Item {
    int node;
    int64_t last;   // packed position of the parent's last token, -1 under the root
    int32_t depth;
  };
  std::vector<Item> stack{{0, -1, 0}};
  while (!stack.empty()) {
    const Item it = stack.back();
    stack.pop_back();
    const Node& n = nodes[it.node];
    int64_t prev = it.last;
    int32_t depth = it.depth;
    for (size_t i = 0; i < n.content.size(); ++i) {
      const int64_t p = npos++;
      if (write) {
        o->token[p] = n.content[i];
        o->parent[p] = (int32_t)prev;
        o->depth[p] = depth;
      }
      if (prev >= 0) {
        const int64_t q = nrows++;
        if (write) {
          o->row_src[q] = (int32_t)prev;
          o->row_target[q] = n.content[i];
          o->row_mask[q] = n.mask[i];
        }
      }
      prev = p;
      ++depth;
    }
    // children in first-seen order: push in reverse
    for (size_t i = n.children.size(); i-- > 0;) stack.push_back({n.children[i], prev, depth});
  }
}

}  // namespace
}  // namespace rlk

using namespace rlk;

extern "C" rlk_status_t rlk_tree_pack(const rlk_calls_t* calls, rlk_tree_out_t* out) {
  if (!calls || !out) return report_error(RLK_EINVAL, "calls or out is NULL");
  const int R = calls->R;
  if (R < 0) return report_error(RLK_ESHAPE, "R < 0");
  if (R > 0 && !calls->call_off) return report_error(RLK_EINVAL, "call_off is NULL");
  const int64_t C = R > 0 ? calls->call_off[R] : 0;
  if (R > 0 && calls->call_off[0] != 0) return report_error(RLK_EINVAL, "call_off[0] must be 0");
  for (int r = 0; r < R; ++r)
    if (calls->call_off[r + 1] < calls->call_off[r]) return report_error(RLK_EINVAL, "call_off decreases");
  if (C > 0 && (!calls->x_off || !calls->y_off)) return report_error(RLK_EINVAL, "x_off or y_off is NULL");
  for (int64_t k = 0; k < C; ++k)
    if (calls->x_off[k + 1] < calls->x_off[k] || calls->y_off[k + 1] < calls->y_off[k])
      return report_error(RLK_EINVAL, "x_off or y_off decreases");
  if (C > 0 && ((calls->x_off[C] > calls->x_off[0] && !calls->x_tok) || (calls->y_off[C] > calls->y_off[0] && !calls->y_tok)))
    return report_error(RLK_EINVAL, "token arrays are NULL");
  const bool query = !out->token && !out->parent && !out->depth && !out->pos_off && !out->row_src &&
                     !out->row_target && !out->row_mask && !out->row_cu && !out->leaves;
  if (!query && (!out->token || !out->parent || !out->depth || !out->pos_off || !out->row_src || !out->row_target ||
                 !out->row_mask || !out->row_cu))
    return report_error(RLK_EINVAL, "some output arrays are NULL (all NULL = size query)");
  // pass 1: sizes
  std::vector<Node> nodes;
  int64_t npos = 0, nrows = 0;
  for (int r = 0; r < R; ++r) {
    build_tree(calls, r, nodes);
    pack_tree(nodes, out, false, npos, nrows);
  }
  out->n_pos = npos;
  out->n_rows = nrows;
  if (query) return RLK_OK;
  if (npos > out->cap_pos || nrows > out->cap_rows) return report_error(RLK_ESHAPE, "output capacity too small");
  if (npos > INT32_MAX || nrows > INT32_MAX) return report_error(RLK_ESHAPE, "more than 2^31 packed positions");
  // pass 2: fill
  npos = nrows = 0;
  out->pos_off[0] = 0;
  out->row_cu[0] = 0;
  for (int r = 0; r < R; ++r) {
    build_tree(calls, r, nodes);
    pack_tree(nodes, out, true, npos, nrows);
    out->pos_off[r + 1] = npos;
    out->row_cu[r + 1] = (int32_t)nrows;
    if (out->leaves) {
      int leaves = 0;
      for (size_t k = 1; k < nodes.size(); ++k) leaves += nodes[k].children.empty();
      out->leaves[r] = leaves;
    }
  }
  return RLK_OK;
}

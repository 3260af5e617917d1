// Graph sharding (paper Sec. 4.2, Alg. 1 and Alg. 2), host code behind the C
// ABI (include/merak_stage.h documents the arguments and the readings taken).
//
// One pass over the nodes in topological order.  State per node: its subgraph
// (sub), for graph inputs their first user (first_user), for common nodes the
// uses still ahead (uses_left), and which subgraph lists it as an output
// (out_of).  Per subgraph: its parameter total, kept up to date as nodes move
// (so the threshold test costs O(1)), and its output list.  A merge into an
// older subgraph walks the visit list back to the dependency, so the pass is
// O(nodes + argument entries + nodes moved).
#include <stdint.h>

#include <vector>

#include "merak_stage.h"

namespace {

struct Sharder {
  int n;
  const int32_t* kind;
  const int64_t* params;
  const int32_t* arg_ptr;
  const int32_t* arg_idx;

  std::vector<int32_t> sub;         // subgraph of a visited node, -1 otherwise
  std::vector<int32_t> first_user;  // graph input -> first node that reads it
  std::vector<int64_t> uses_left;   // common node -> remaining uses
  std::vector<int32_t> out_of;      // node -> subgraph whose outputs list it, -1
  std::vector<int32_t> visited;     // N: visit order
  std::vector<double> psum;         // subgraph -> parameter total
  std::vector<std::vector<int32_t>> outs;  // subgraph -> outputs (closed subgraphs)

  // Alg. 1 for node i in current subgraph s: the smallest subgraph it may join
  // and the node that forces it (-1 if none).  Updates uses_left/first_user.
  void dependency(int i, int s, int* s_min, int* n_min) {
    *s_min = s;
    *n_min = -1;
    const int last = visited.empty() ? -1 : visited.back();
    for (int e = arg_ptr[i]; e < arg_ptr[i + 1]; ++e) {
      const int a = arg_idx[e];
      if (kind[a] == MERAK_NODE_COMMON) {
        --uses_left[a];
      } else if (kind[a] == MERAK_NODE_INPUT) {
        if (first_user[a] < 0) {
          first_user[a] = i;
        } else if (first_user[a] != i && sub[first_user[a]] < *s_min) {  // a second read by i itself: none
          *s_min = sub[first_user[a]];
          *n_min = first_user[a];
        }
      } else if (out_of[a] >= 0) {
        if (sub[a] + 1 < *s_min) {
          *s_min = sub[a] + 1;
          *n_min = a;
        }
      } else if (sub[a] >= 0 && a != last) {
        if (sub[a] < *s_min) {
          *s_min = sub[a];
          *n_min = a;
        }
      }
    }
  }

  void drop_outputs_from(int t) {  // subgraphs t, t+1, ... are open again / gone
    for (int u = t; u < (int)outs.size(); ++u)
      for (int o : outs[u])
        if (out_of[o] == u) out_of[o] = -1;
    if ((int)outs.size() > t) outs.resize(t);
  }

  int run(int k) {
    sub.assign(n, -1);
    first_user.assign(n, -1);
    uses_left.assign(n, 0);
    out_of.assign(n, -1);
    double total = 0.0;
    for (int i = 0; i < n; ++i) total += (double)params[i];
    for (int i = 0; i < n; ++i)
      for (int e = arg_ptr[i]; e < arg_ptr[i + 1]; ++e)
        if (kind[arg_idx[e]] == MERAK_NODE_COMMON) ++uses_left[arg_idx[e]];
    const double p = total / (double)k;
    psum.assign(1, 0.0);
    int s = 0;
    for (int i = 0; i < n; ++i) {
      if (kind[i] == MERAK_NODE_INPUT) continue;
      int s_min, n_min;
      dependency(i, s, &s_min, &n_min);
      if (s_min < s) {
        s = s_min;
        for (int v = (int)visited.size() - 1; v >= 0 && visited[v] != n_min; --v) {
          const int m = visited[v];
          psum[sub[m]] -= (double)params[m];
          sub[m] = s;
          psum[s] += (double)params[m];
        }
        drop_outputs_from(s);
      }
      sub[i] = s;
      visited.push_back(i);
      if ((int)psum.size() <= s) psum.resize(s + 1, 0.0);
      psum[s] += (double)params[i];
      if (psum[s] > p) {  // close subgraph s
        if ((int)outs.size() <= s) outs.resize(s + 1);
        std::vector<int32_t>& o = outs[s];
        o.clear();
        for (int m : visited)  // visited common nodes with uses left, in visit order
          if (kind[m] == MERAK_NODE_COMMON && uses_left[m] > 0) o.push_back(m);
        o.push_back(i);
        for (int m : o)
          if (kind[m] != MERAK_NODE_COMMON) out_of[m] = s;
        ++s;
        if ((int)psum.size() <= s) psum.resize(s + 1, 0.0);
      }
    }
    int last = -1;
    for (int m : visited) last = sub[m] > last ? sub[m] : last;
    return last + 1;
  }
};

bool check_graph(int n, const int32_t* kind, const int64_t* params, const int32_t* arg_ptr, const int32_t* arg_idx,
                 const int32_t* common_uses) {
  if (arg_ptr[0] != 0) return false;
  for (int i = 0; i < n; ++i) {
    if (kind[i] < MERAK_NODE_COMPUTE || kind[i] > MERAK_NODE_COMMON) return false;
    if (params[i] < 0 || arg_ptr[i + 1] < arg_ptr[i]) return false;
    if (kind[i] == MERAK_NODE_INPUT && arg_ptr[i + 1] != arg_ptr[i]) return false;
    if (kind[i] == MERAK_NODE_COMMON && common_uses[i] < 0) return false;
    for (int e = arg_ptr[i]; e < arg_ptr[i + 1]; ++e)
      if (arg_idx[e] < 0 || arg_idx[e] >= i) return false;
  }
  // the use counts given for common nodes must be the counts in arg_idx
  std::vector<int64_t> uses(n, 0);
  for (int e = 0; e < arg_ptr[n]; ++e) ++uses[arg_idx[e]];
  for (int i = 0; i < n; ++i)
    if (kind[i] == MERAK_NODE_COMMON && uses[i] != common_uses[i]) return false;
  return true;
}

}  // namespace

extern "C" int merak_graph_shard(int n_nodes, const int32_t* kind, const int64_t* params, const int32_t* arg_ptr,
                                 const int32_t* arg_idx, const int32_t* common_uses, int n_outputs,
                                 const int32_t* graph_outputs, int k, int32_t* subgraph_of, int32_t* n_subgraphs,
                                 int32_t* io_ptr, int32_t* io_idx, int io_capacity) {
  if (n_nodes < 1 || k < 1 || n_outputs < 0 || io_capacity < 0) return MERAK_ERR_INVALID_ARG;
  if (!kind || !params || !arg_ptr || !common_uses || !subgraph_of || !n_subgraphs || !io_ptr) return MERAK_ERR_INVALID_ARG;
  if ((arg_ptr[n_nodes] > 0 && !arg_idx) || (n_outputs > 0 && !graph_outputs) || (io_capacity > 0 && !io_idx))
    return MERAK_ERR_INVALID_ARG;
  if (!check_graph(n_nodes, kind, params, arg_ptr, arg_idx, common_uses)) return MERAK_ERR_INVALID_ARG;
  for (int j = 0; j < n_outputs; ++j)
    if (graph_outputs[j] < 0 || graph_outputs[j] >= n_nodes || kind[graph_outputs[j]] == MERAK_NODE_INPUT)
      return MERAK_ERR_INVALID_ARG;

  Sharder sh{n_nodes, kind, params, arg_ptr, arg_idx, {}, {}, {}, {}, {}, {}, {}};
  const int S = sh.run(k);
  for (int i = 0; i < n_nodes; ++i) subgraph_of[i] = sh.sub[i];
  *n_subgraphs = S;

  // Inputs: the previous subgraph's outputs, then the graph inputs whose first
  // user is here (in index order).  Outputs: the recorded list, or the graph
  // outputs for the last subgraph.
  std::vector<std::vector<int32_t>> graph_in(S);
  for (int x = 0; x < n_nodes; ++x)
    if (kind[x] == MERAK_NODE_INPUT && sh.first_user[x] >= 0) graph_in[sh.sub[sh.first_user[x]]].push_back(x);
  int pos = 0;
  bool fits = true;
  auto put = [&](int32_t v) {
    if (pos < io_capacity) io_idx[pos] = v;
    else fits = false;
    ++pos;
  };
  for (int j = 0; j < S; ++j) {
    io_ptr[2 * j] = pos;
    if (j > 0 && j - 1 < (int)sh.outs.size())
      for (int o : sh.outs[j - 1]) put(o);
    for (int x : graph_in[j]) put(x);
    io_ptr[2 * j + 1] = pos;
    if (j < S - 1) {
      if (j < (int)sh.outs.size())
        for (int o : sh.outs[j]) put(o);
    } else {
      for (int q = 0; q < n_outputs; ++q) put(graph_outputs[q]);
    }
  }
  io_ptr[2 * S] = pos;
  return fits ? MERAK_OK : MERAK_ERR_WORKSPACE;
}

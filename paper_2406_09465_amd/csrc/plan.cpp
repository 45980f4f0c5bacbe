// Plan validation (Korch, Definitions 1 and 3; output and dependency
// constraints of Section 4.2 with an explicit kernel order), the unfused
// plan, the state search of Algorithm 1, and workspace planning.
#include "plan.h"

#include <algorithm>
#include <set>

namespace korch {

int resolve_storage(const Graph& g, const std::vector<KernelDesc>& ks, int k, int u) {
  int v = u;
  while (true) {
    if (g.nodes[v].op == KORCH_INPUT) return v;
    for (int j = 0; j < k; ++j)
      if (std::binary_search(ks[j].outs.begin(), ks[j].outs.end(), v)) return v;
    if (g.is_view(v))
      v = g.nodes[v].in[0];
    else
      return -1;
  }
}

void validate_plan(const Graph& g, const std::vector<KernelDesc>& ks, bool strict) {
  if (!g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
  if (ks.empty()) fail(KORCH_E_PLAN_EMPTY, "plan has no kernels");
  int n = (int)g.nodes.size();
  for (size_t k = 0; k < ks.size(); ++k) {
    const KernelDesc& kd = ks[k];
    std::string where = "kernel " + std::to_string(k) + ": ";
    if (kd.prims.empty()) fail(KORCH_E_PLAN_EMPTY, where + "no primitives");
    for (size_t i = 0; i < kd.prims.size(); ++i) {
      int v = kd.prims[i];
      if (v < 0 || v >= n) fail(KORCH_E_ARG, where + "node id out of range");
      if (!g.is_prim(v)) fail(KORCH_E_PLAN_EMPTY, where + "contains graph input " + std::to_string(v));
      if (i && kd.prims[i - 1] == v) fail(KORCH_E_ARG, where + "duplicate node");
    }
    if (!is_convex(g, kd.prims)) fail(KORCH_E_PLAN_NONCONVEX, where + "primitive set is not convex (Definition 1)");
    if (kd.outs.empty()) fail(KORCH_E_PLAN_BAD_OUTPUT, where + "empty output set");
    if (strict && kd.outs.size() != 1)
      fail(KORCH_E_PLAN_MULTI_OUTPUT, where + "more than one output while single-output mode is on");
    std::set<int> in(kd.prims.begin(), kd.prims.end());
    for (size_t i = 0; i < kd.outs.size(); ++i) {
      int o = kd.outs[i];
      if (o < 0 || o >= n || !in.count(o)) fail(KORCH_E_PLAN_BAD_OUTPUT, where + "output not in the kernel");
      if (i && kd.outs[i - 1] == o) fail(KORCH_E_ARG, where + "duplicate output");
      bool external = g.is_output(o);
      for (int c : g.consumers[o])
        if (!in.count(c)) external = true;
      if (!external)
        fail(KORCH_E_PLAN_BAD_OUTPUT,
             where + "output " + std::to_string(o) + " has no consumer outside the kernel (Definition 3)");
    }
    for (int u : external_inputs(g, kd))
      if (resolve_storage(g, ks, (int)k, u) < 0)
        fail(KORCH_E_PLAN_DEP_ORDER, where + "reads node " + std::to_string(u) + ", which no earlier kernel materializes");
  }
  for (int o : g.outputs) {
    bool covered = false;
    for (auto& kd : ks)
      if (std::binary_search(kd.outs.begin(), kd.outs.end(), o)) covered = true;
    if (!covered) fail(KORCH_E_PLAN_OUTPUT_UNCOVERED, "graph output " + std::to_string(o) + " is never materialized");
  }
}

std::vector<KernelDesc> unfused_plan(const Graph& g) {
  std::vector<KernelDesc> ks;
  int n = (int)g.nodes.size();
  // A reshape whose source is available is a view: no kernel, unless the
  // reshape itself is a graph output.
  for (int v = 0; v < n; ++v) {
    if (!g.is_prim(v)) continue;
    if (g.is_view(v) && !g.is_output(v)) continue;
    KernelDesc kd;
    kd.prims = {v};
    kd.outs = {v};
    ks.push_back(kd);
  }
  return ks;
}

std::vector<Bits> execution_states(const Graph& g, size_t max_states) {
  int n = (int)g.nodes.size();
  std::vector<int> prims;
  for (int v = 0; v < n; ++v)
    if (g.is_prim(v)) prims.push_back(v);
  std::set<Bits> seen;
  std::vector<Bits> order;
  std::vector<Bits> stack;
  Bits empty(n);
  seen.insert(empty);
  order.push_back(empty);
  stack.push_back(empty);
  while (!stack.empty()) {
    Bits x = stack.back();
    stack.pop_back();
    for (int v : prims) {
      if (x.test(v)) continue;
      bool ready = true;
      for (int u : g.nodes[v].in)
        if (g.is_prim(u) && !x.test(u)) ready = false;
      if (!ready) continue;
      Bits x2 = x;
      x2.set(v);
      if (seen.insert(x2).second) {
        if (seen.size() > max_states) fail(KORCH_E_ARG, "more execution states than the limit");
        order.push_back(x2);
        stack.push_back(x2);
      }
    }
  }
  return order;
}

void plan_workspace(Plan& p) {
  const Graph& g = p.g;
  auto& ks = p.kernels;
  int K = (int)ks.size();
  struct Item {
    size_t bytes;
    int first, last;
    int node;      // >= 0: materialized tensor
    int kernel;    // scratch owner when node < 0
    int argi;
    size_t off = 0;
  };
  std::vector<Item> items;
  std::map<int, int> item_of;
  for (int k = 0; k < K; ++k)
    for (int o : ks[k].outs) {
      if (g.is_output(o)) continue;
      auto it = item_of.find(o);
      if (it == item_of.end()) {
        item_of[o] = (int)items.size();
        items.push_back({(size_t)numel(g.nodes[o].shape) * dtype_bytes(g.nodes[o].dtype), k, k, o, -1, -1});
      } else {
        items[it->second].last = std::max(items[it->second].last, k);
      }
    }
  for (int k = 0; k < K; ++k)
    for (int u : external_inputs(g, ks[k])) {
      int s = resolve_storage(g, ks, k, u);
      auto it = item_of.find(s);
      if (it != item_of.end()) items[it->second].last = std::max(items[it->second].last, k);
    }
  p.counter_bytes = 0;
  for (int k = 0; k < (int)p.ck.size(); ++k) {
    auto& args = p.ck[k].gen.args;
    for (int a = 0; a < (int)args.size(); ++a) {
      if (args[a].kind == ArgRef::Scratch) items.push_back({args[a].bytes, k, k, -1, k, a});
      if (args[a].kind == ArgRef::Counter) {
        Storage s;
        s.kind = Storage::Counters;
        s.offset = p.counter_bytes;
        p.counter_bytes += (args[a].bytes + 255) / 256 * 256;
        p.ck[k].arg_storage.resize(args.size());
        p.ck[k].arg_storage[a] = s;
      }
    }
  }
  // First fit over (time interval x address range), largest first.
  std::vector<int> order(items.size());
  for (size_t i = 0; i < items.size(); ++i) order[i] = (int)i;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    if (items[a].bytes != items[b].bytes) return items[a].bytes > items[b].bytes;
    return items[a].first < items[b].first;
  });
  std::vector<int> placed;
  size_t total = 0;
  for (int i : order) {
    Item& it = items[i];
    size_t sz = (it.bytes + 255) / 256 * 256;
    std::vector<std::pair<size_t, size_t>> busy;
    for (int j : placed) {
      const Item& o = items[j];
      if (o.last < it.first || it.last < o.first) continue;
      busy.push_back({o.off, o.off + (o.bytes + 255) / 256 * 256});
    }
    std::sort(busy.begin(), busy.end());
    size_t off = 0;
    for (auto& b : busy) {
      if (off + sz <= b.first) break;
      off = std::max(off, b.second);
    }
    it.off = off;
    placed.push_back(i);
    total = std::max(total, off + sz);
  }
  p.ws_bytes = total;
  p.ws_offset.clear();
  for (auto& it : items) {
    if (it.node >= 0) {
      p.ws_offset[it.node] = it.off;
    } else {
      Storage s;
      s.kind = Storage::Workspace;
      s.offset = it.off;
      p.ck[it.kernel].arg_storage.resize(p.ck[it.kernel].gen.args.size());
      p.ck[it.kernel].arg_storage[it.argi] = s;
    }
  }
  // Tensor / output arguments.
  for (int k = 0; k < (int)p.ck.size(); ++k) {
    auto& ck = p.ck[k];
    ck.arg_storage.resize(ck.gen.args.size());
    for (size_t a = 0; a < ck.gen.args.size(); ++a) {
      const ArgRef& r = ck.gen.args[a];
      if (r.kind != ArgRef::Tensor && r.kind != ArgRef::Output) continue;
      int s = r.kind == ArgRef::Tensor ? resolve_storage(g, ks, k, r.node) : r.node;
      if (s < 0) fail(KORCH_E_PLAN_DEP_ORDER, "internal: unresolved tensor argument");
      Storage st;
      if (g.nodes[s].op == KORCH_INPUT) {
        st.kind = Storage::GraphInput;
        st.index = (int)(std::find(g.inputs.begin(), g.inputs.end(), s) - g.inputs.begin());
      } else if (g.is_output(s)) {
        st.kind = Storage::GraphOutput;
        st.index = (int)(std::find(g.outputs.begin(), g.outputs.end(), s) - g.outputs.begin());
      } else {
        st.kind = Storage::Workspace;
        st.offset = p.ws_offset.at(s);
      }
      ck.arg_storage[a] = st;
    }
  }
}

}  // namespace korch

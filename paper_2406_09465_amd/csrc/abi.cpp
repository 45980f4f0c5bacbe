// extern "C" boundary: status codes, thread-local error text, no exceptions
// across the ABI.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <set>

#include "plan.h"

using namespace korch;

struct korch_graph {
  Graph g;
};
struct korch_plan {
  Plan p;
};

namespace korch {
Graph rewrite_graph(const Graph& g, uint32_t rules, int* applied);
void compile_plan(Plan& p);
void generate_plan(Plan& p);
void load_plan(Plan& p);
void destroy_plan_device(Plan& p);
void execute_plan(Plan& p, const void* const* inputs, void* const* outputs, void* ws, size_t ws_bytes,
                  hipStream_t stream, int first, int count, void* const* starts = nullptr,
                  void* const* stops = nullptr, void* counters = nullptr);
void execute_plan_noalloc(Plan& p, const void* const* inputs, void* const* outputs, hipStream_t stream);
void compile_candidate(const Graph& g, const KernelDesc& kd);
void flush_caches(void* buf, size_t bytes, int write, hipStream_t stream);
float profile_candidate(const Graph& g, const KernelDesc& kd, int warmup, int reps, size_t flush_bytes,
                        hipStream_t stream);
}  // namespace korch

static thread_local std::string g_err;

template <typename F>
static int guard(F&& f) {
  try {
    f();
    g_err.clear();
    return KORCH_OK;
  } catch (Error& e) {
    g_err = e.what();
    return e.code;
  } catch (std::bad_alloc&) {
    g_err = "out of host memory";
    return KORCH_E_ARG;
  } catch (std::exception& e) {
    g_err = e.what();
    return KORCH_E_ARG;
  } catch (...) {
    g_err = "unknown error";
    return KORCH_E_ARG;
  }
}

#define NEED(x)                                        \
  do {                                                 \
    if (!(x)) fail(KORCH_E_ARG, "NULL argument: " #x); \
  } while (0)

static bool strict_mode() {
  const char* s = getenv("KORCH_STRICT_SINGLE_OUTPUT");
  return s && *s && strcmp(s, "0") != 0;
}

static KernelDesc to_desc(const korch_kernel_desc& k) {
  if (k.n_prims < 0 || k.n_outs < 0) fail(KORCH_E_ARG, "negative count");
  if ((k.n_prims && !k.prims) || (k.n_outs && !k.outs)) fail(KORCH_E_ARG, "NULL id array");
  KernelDesc d;
  d.prims.assign(k.prims, k.prims + k.n_prims);
  d.outs.assign(k.outs, k.outs + k.n_outs);
  std::sort(d.prims.begin(), d.prims.end());
  std::sort(d.outs.begin(), d.outs.end());
  return d;
}

extern "C" {

const char* korch_last_error(void) { return g_err.c_str(); }

const char* korch_status_name(int s) {
  switch (s) {
    case KORCH_OK: return "KORCH_OK";
    case KORCH_E_ARG: return "KORCH_E_ARG";
    case KORCH_E_SHAPE: return "KORCH_E_SHAPE";
    case KORCH_E_CYCLE: return "KORCH_E_CYCLE";
    case KORCH_E_STATE: return "KORCH_E_STATE";
    case KORCH_E_PLAN_EMPTY: return "KORCH_E_PLAN_EMPTY";
    case KORCH_E_PLAN_NONCONVEX: return "KORCH_E_PLAN_NONCONVEX";
    case KORCH_E_PLAN_BAD_OUTPUT: return "KORCH_E_PLAN_BAD_OUTPUT";
    case KORCH_E_PLAN_DEP_ORDER: return "KORCH_E_PLAN_DEP_ORDER";
    case KORCH_E_PLAN_OUTPUT_UNCOVERED: return "KORCH_E_PLAN_OUTPUT_UNCOVERED";
    case KORCH_E_PLAN_MULTI_OUTPUT: return "KORCH_E_PLAN_MULTI_OUTPUT";
    case KORCH_E_UNSUPPORTED: return "KORCH_E_UNSUPPORTED";
    case KORCH_E_ALIGN: return "KORCH_E_ALIGN";
    case KORCH_E_WORKSPACE: return "KORCH_E_WORKSPACE";
    case KORCH_E_COMPILE: return "KORCH_E_COMPILE";
    case KORCH_E_HIP: return "KORCH_E_HIP";
  }
  return "KORCH_E_UNKNOWN";
}

int korch_graph_create(korch_graph** g) {
  return guard([&] {
    NEED(g);
    *g = new korch_graph();
  });
}

void korch_graph_destroy(korch_graph* g) { delete g; }

int korch_graph_input(korch_graph* g, korch_dtype dtype, int32_t rank, const int64_t* shape, int32_t* node) {
  return guard([&] {
    NEED(g);
    NEED(node);
    if (rank < 0 || rank > KORCH_MAX_RANK || (rank && !shape)) fail(KORCH_E_ARG, "bad rank or shape");
    *node = g->g.add_input(dtype, Shape(shape, shape + rank));
  });
}

int korch_graph_op(korch_graph* g, korch_op op, int32_t n_in, const int32_t* in, const korch_attrs* attrs,
                   korch_dtype out_dtype, int32_t* node) {
  return guard([&] {
    NEED(g);
    NEED(node);
    if (n_in < 0 || (n_in && !in)) fail(KORCH_E_ARG, "bad input list");
    std::vector<int> ins(in, in + n_in);
    if (op == KORCH_RESHAPE && n_in == 1 && ins[0] >= 0 && ins[0] < (int)g->g.nodes.size() &&
        g->g.nodes[ins[0]].dtype != (int)out_dtype)
      fail(KORCH_E_ARG, "reshape must keep its input's dtype");
    *node = g->g.add_op(op, ins, attrs, out_dtype);
  });
}

int korch_graph_output(korch_graph* g, int32_t node) {
  return guard([&] {
    NEED(g);
    g->g.add_output(node);
  });
}

int korch_graph_finalize(korch_graph* g) {
  return guard([&] {
    NEED(g);
    g->g.finalize();
  });
}

int korch_graph_num_nodes(const korch_graph* g, int32_t* n) {
  return guard([&] {
    NEED(g);
    NEED(n);
    *n = (int32_t)g->g.nodes.size();
  });
}

int korch_graph_node_attrs(const korch_graph* g, int32_t node, korch_attrs* attrs) {
  return guard([&] {
    NEED(g);
    NEED(attrs);
    if (node < 0 || node >= (int)g->g.nodes.size()) fail(KORCH_E_ARG, "node id out of range");
    const Node& n = g->g.nodes[node];
    *attrs = n.attrs;
    if (op_kind(n.op) == Kind::Reduce || n.op == KORCH_CONCAT) attrs->axis = n.axis;
  });
}

int korch_graph_rewrite(const korch_graph* g, uint32_t rules, korch_graph** out, int32_t* applied) {
  return guard([&] {
    NEED(g);
    NEED(out);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    int n = 0;
    korch_graph* r = new korch_graph();
    try {
      r->g = rewrite_graph(g->g, rules, &n);
    } catch (...) {
      delete r;
      throw;
    }
    *out = r;
    if (applied) *applied = n;
  });
}

int korch_graph_node_info(const korch_graph* g, int32_t node, int32_t* op, int32_t* dtype, int32_t* rank,
                          int64_t* shape) {
  return guard([&] {
    NEED(g);
    if (node < 0 || node >= (int)g->g.nodes.size()) fail(KORCH_E_ARG, "node id out of range");
    const Node& n = g->g.nodes[node];
    if (op) *op = n.op;
    if (dtype) *dtype = n.dtype;
    if (rank) *rank = (int32_t)n.shape.size();
    if (shape)
      for (size_t i = 0; i < n.shape.size(); ++i) shape[i] = n.shape[i];
  });
}

int korch_graph_node_inputs(const korch_graph* g, int32_t node, int32_t* ids, int32_t cap, int32_t* n) {
  return guard([&] {
    NEED(g);
    NEED(n);
    if (node < 0 || node >= (int)g->g.nodes.size()) fail(KORCH_E_ARG, "node id out of range");
    if (cap < 0 || (cap > 0 && !ids)) fail(KORCH_E_ARG, "bad id buffer");
    const auto& in = g->g.nodes[node].in;
    *n = (int32_t)in.size();
    for (int i = 0; i < (int)in.size() && i < cap; ++i) ids[i] = in[i];
  });
}

int korch_graph_num_inputs(const korch_graph* g, int32_t* n) {
  return guard([&] {
    NEED(g);
    NEED(n);
    *n = (int32_t)g->g.inputs.size();
  });
}

int korch_graph_num_outputs(const korch_graph* g, int32_t* n) {
  return guard([&] {
    NEED(g);
    NEED(n);
    *n = (int32_t)g->g.outputs.size();
  });
}

int korch_graph_input_node(const korch_graph* g, int32_t i, int32_t* node) {
  return guard([&] {
    NEED(g);
    NEED(node);
    if (i < 0 || i >= (int)g->g.inputs.size()) fail(KORCH_E_ARG, "input index out of range");
    *node = g->g.inputs[i];
  });
}

int korch_graph_output_node(const korch_graph* g, int32_t i, int32_t* node) {
  return guard([&] {
    NEED(g);
    NEED(node);
    if (i < 0 || i >= (int)g->g.outputs.size()) fail(KORCH_E_ARG, "output index out of range");
    *node = g->g.outputs[i];
  });
}

int korch_is_convex(const korch_graph* g, int32_t n, const int32_t* nodes, int32_t* convex) {
  return guard([&] {
    NEED(g);
    NEED(convex);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    if (n < 0 || (n && !nodes)) fail(KORCH_E_ARG, "bad node list");
    std::vector<int> v(nodes, nodes + n);
    for (int x : v)
      if (x < 0 || x >= (int)g->g.nodes.size()) fail(KORCH_E_ARG, "node id out of range");
    *convex = is_convex(g->g, v) ? 1 : 0;
  });
}

int korch_enumerate_states(const korch_graph* g, int32_t max_states,
                           int (*cb)(const uint8_t* member, int32_t n_nodes, void* user), void* user) {
  return guard([&] {
    NEED(g);
    NEED(cb);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    auto states = execution_states(g->g, (size_t)std::max(1, max_states));
    int n = (int)g->g.nodes.size();
    std::vector<uint8_t> mem(n);
    for (auto& s : states) {
      for (int i = 0; i < n; ++i) mem[i] = s.test(i) ? 1 : 0;
      if (cb(mem.data(), n, user)) break;
    }
  });
}

int korch_kernel_family(const korch_graph* g, const korch_kernel_desc* k, int32_t* family) {
  return guard([&] {
    NEED(g);
    NEED(k);
    NEED(family);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    std::string why;
    *family = match_family(g->g, to_desc(*k), &why);
    if (*family == KORCH_FAM_NONE) g_err = why;
  });
}

int korch_enumerate_candidates(const korch_graph* g, int32_t max_prims, int32_t max_outs, int32_t only_supported,
                               int (*cb)(const korch_kernel_desc* k, void* user), void* user) {
  return guard([&] {
    NEED(g);
    NEED(cb);
    const Graph& G = g->g;
    if (!G.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    auto states = execution_states(G, 100000);
    int n = (int)G.nodes.size();
    std::set<std::vector<int>> seen;
    for (auto& d1 : states)
      for (auto& d2 : states) {
        if (d1 == d2 || !d1.subset_of(d2)) continue;
        std::vector<int> pr;
        for (int i = 0; i < n; ++i)
          if (d2.test(i) && !d1.test(i)) pr.push_back(i);
        if ((int)pr.size() > max_prims || !seen.insert(pr).second) continue;
        std::set<int> in(pr.begin(), pr.end());
        std::vector<int> omax;
        for (int v : pr) {
          bool ext = G.is_output(v);
          for (int c : G.consumers[v])
            if (!in.count(c)) ext = true;
          if (ext) omax.push_back(v);
        }
        if (omax.empty()) continue;
        std::vector<std::vector<int>> osets;
        int m = (int)omax.size();
        if (m <= max_outs) {
          for (int mask = 1; mask < (1 << m); ++mask) {
            std::vector<int> o;
            for (int i = 0; i < m; ++i)
              if (mask >> i & 1) o.push_back(omax[i]);
            osets.push_back(o);
          }
        } else {
          osets.push_back(omax);
          for (int v : omax) osets.push_back({v});
        }
        for (auto& o : osets) {
          KernelDesc kd{pr, o};
          if (only_supported) {
            std::string why;
            if (match_family(G, kd, &why) == KORCH_FAM_NONE) continue;
          }
          korch_kernel_desc d{(int32_t)pr.size(), pr.data(), (int32_t)o.size(), o.data()};
          if (cb(&d, user)) return;
        }
      }
  });
}

int korch_plan_create(const korch_graph* g, int32_t n_kernels, const korch_kernel_desc* kernels, korch_plan** p) {
  return guard([&] {
    NEED(g);
    NEED(p);
    if (n_kernels < 0 || (n_kernels && !kernels)) fail(KORCH_E_ARG, "bad kernel list");
    std::vector<KernelDesc> ks;
    for (int i = 0; i < n_kernels; ++i) ks.push_back(to_desc(kernels[i]));
    validate_plan(g->g, ks, strict_mode());
    auto* q = new korch_plan();
    q->p.g = g->g;
    q->p.kernels = ks;
    *p = q;
  });
}

int korch_plan_unfused(const korch_graph* g, korch_plan** p) {
  return guard([&] {
    NEED(g);
    NEED(p);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    auto ks = unfused_plan(g->g);
    validate_plan(g->g, ks, false);
    auto* q = new korch_plan();
    q->p.g = g->g;
    q->p.kernels = ks;
    q->p.name_prefix = "korch_u";
    *p = q;
  });
}

void korch_plan_destroy(korch_plan* p) {
  if (!p) return;
  try {
    destroy_plan_device(p->p);
  } catch (...) {
  }
  delete p;
}

int korch_plan_num_kernels(const korch_plan* p, int32_t* n) {
  return guard([&] {
    NEED(p);
    NEED(n);
    *n = (int32_t)p->p.kernels.size();
  });
}

int korch_plan_compile(korch_plan* p) {
  return guard([&] {
    NEED(p);
    compile_plan(p->p);
  });
}

int korch_plan_load(korch_plan* p) {
  return guard([&] {
    NEED(p);
    load_plan(p->p);
  });
}

int korch_plan_workspace_bytes(const korch_plan* p, size_t* bytes) {
  return guard([&] {
    NEED(p);
    NEED(bytes);
    generate_plan(const_cast<Plan&>(p->p));
    *bytes = p->p.ws_bytes;
  });
}

int korch_plan_execute(korch_plan* p, const void* const* inputs, void* const* outputs, void* workspace,
                       size_t workspace_bytes, void* stream) {
  return guard([&] {
    NEED(p);
    execute_plan(p->p, inputs, outputs, workspace, workspace_bytes, (hipStream_t)stream, 0, -1);
  });
}

int korch_plan_execute_noalloc(korch_plan* p, const void* const* inputs, void* const* outputs, void* stream) {
  return guard([&] {
    NEED(p);
    execute_plan_noalloc(p->p, inputs, outputs, (hipStream_t)stream);
  });
}

int korch_plan_execute_kernels(korch_plan* p, int32_t first, int32_t count, const void* const* inputs,
                               void* const* outputs, void* workspace, size_t workspace_bytes, void* stream) {
  return guard([&] {
    NEED(p);
    if (count < 0) fail(KORCH_E_ARG, "negative kernel count");
    execute_plan(p->p, inputs, outputs, workspace, workspace_bytes, (hipStream_t)stream, first, count);
  });
}

int korch_plan_execute_timed(korch_plan* p, int32_t first, int32_t count, const void* const* inputs,
                             void* const* outputs, void* workspace, size_t workspace_bytes, void* stream, int32_t timed,
                             void* start, void* stop) {
  return guard([&] {
    NEED(p);
    if (count < 0) fail(KORCH_E_ARG, "negative kernel count");
    if (timed < first || timed >= first + count) fail(KORCH_E_ARG, "timed kernel outside the launched range");
    std::vector<void*> starts(p->p.kernels.size(), nullptr), stops(p->p.kernels.size(), nullptr);
    if (timed >= 0 && timed < (int)starts.size()) {
      starts[timed] = start;
      stops[timed] = stop;
    }
    execute_plan(p->p, inputs, outputs, workspace, workspace_bytes, (hipStream_t)stream, first, count, starts.data(),
                 stops.data());
  });
}

int korch_plan_execute_events(korch_plan* p, const void* const* inputs, void* const* outputs, void* workspace,
                              size_t workspace_bytes, void* stream, void* const* start_events,
                              void* const* stop_events) {
  return guard([&] {
    NEED(p);
    execute_plan(p->p, inputs, outputs, workspace, workspace_bytes, (hipStream_t)stream, 0, -1, start_events,
                 stop_events);
  });
}

int korch_plan_kernel_info(const korch_plan* p, int32_t k, int32_t* family, double* alg_bytes, double* alg_flops) {
  return guard([&] {
    NEED(p);
    generate_plan(const_cast<Plan&>(p->p));
    if (k < 0 || k >= (int)p->p.ck.size()) fail(KORCH_E_ARG, "kernel index out of range");
    const GenKernel& gk = p->p.ck[k].gen;
    if (family) *family = gk.family;
    if (alg_bytes) *alg_bytes = gk.alg_bytes;
    if (alg_flops) *alg_flops = gk.alg_flops;
  });
}

int korch_kernel_source(const korch_graph* g, const korch_kernel_desc* k, char* buf, size_t cap, size_t* len) {
  return guard([&] {
    NEED(g);
    NEED(k);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    KernelDesc d = to_desc(*k);
    if (d.prims.empty() || d.outs.empty()) fail(KORCH_E_ARG, "empty kernel");
    for (int v : d.prims)
      if (v < 0 || v >= (int)g->g.nodes.size() || !g->g.is_prim(v)) fail(KORCH_E_ARG, "bad primitive id");
    for (int v : d.outs)
      if (std::find(d.prims.begin(), d.prims.end(), v) == d.prims.end()) fail(KORCH_E_ARG, "output outside the kernel");
    std::string s = generate_kernel(g->g, d, 0).source;
    if (len) *len = s.size();
    if (buf && cap) {
      size_t n = std::min(cap - 1, s.size());
      memcpy(buf, s.data(), n);
      buf[n] = 0;
    }
  });
}

int korch_plan_kernel_source(const korch_plan* p, int32_t k, char* buf, size_t cap, size_t* len) {
  return guard([&] {
    NEED(p);
    generate_plan(const_cast<Plan&>(p->p));
    if (k < 0 || k >= (int)p->p.ck.size()) fail(KORCH_E_ARG, "kernel index out of range");
    const std::string& s = p->p.ck[k].gen.source;
    if (len) *len = s.size();
    if (buf && cap) {
      size_t n = std::min(cap - 1, s.size());
      memcpy(buf, s.data(), n);
      buf[n] = 0;
    }
  });
}

int korch_plan_kernel_code(const korch_plan* p, int32_t k, void* buf, size_t cap, size_t* len) {
  return guard([&] {
    NEED(p);
    if (!p->p.compiled) fail(KORCH_E_STATE, "plan is not compiled");
    if (k < 0 || k >= (int)p->p.ck.size()) fail(KORCH_E_ARG, "kernel index out of range");
    const std::vector<char>& c = p->p.ck[k].code;
    if (len) *len = c.size();
    if (buf && cap) memcpy(buf, c.data(), std::min(cap, c.size()));
  });
}

int korch_plan_kernel_name(const korch_plan* p, int32_t k, char* buf, size_t cap) {
  return guard([&] {
    NEED(p);
    NEED(buf);
    generate_plan(const_cast<Plan&>(p->p));
    if (k < 0 || k >= (int)p->p.ck.size()) fail(KORCH_E_ARG, "kernel index out of range");
    const std::string& s = p->p.ck[k].gen.name;
    if (cap == 0) fail(KORCH_E_ARG, "zero capacity");
    size_t n = std::min(cap - 1, s.size());
    memcpy(buf, s.data(), n);
    buf[n] = 0;
  });
}

int korch_plan_kernel_launch(const korch_plan* p, int32_t k, int32_t grid[3], int32_t block[3], int32_t* lds_bytes) {
  return guard([&] {
    NEED(p);
    generate_plan(const_cast<Plan&>(p->p));
    if (k < 0 || k >= (int)p->p.ck.size()) fail(KORCH_E_ARG, "kernel index out of range");
    const GenKernel& gk = p->p.ck[k].gen;
    for (int i = 0; i < 3; ++i) {
      if (grid) grid[i] = gk.grid[i];
      if (block) block[i] = gk.block[i];
    }
    if (lds_bytes) *lds_bytes = gk.lds_bytes;
  });
}

int korch_compile_candidate(const korch_graph* g, const korch_kernel_desc* k) {
  return guard([&] {
    NEED(g);
    NEED(k);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    KernelDesc kd = to_desc(*k);
    std::string why;
    if (match_family(g->g, kd, &why) == KORCH_FAM_NONE) fail(KORCH_E_UNSUPPORTED, why);
    compile_candidate(g->g, kd);
  });
}

int korch_flush_caches(void* buffer, size_t bytes, int32_t write, void* stream) {
  return guard([&] {
    if (bytes && !buffer) fail(KORCH_E_ARG, "null flush buffer");
    if (((uintptr_t)buffer & 15) != 0) fail(KORCH_E_ALIGN, "flush buffer must be 16-byte aligned");
    flush_caches(buffer, bytes, write ? 1 : 0, (hipStream_t)stream);
  });
}

int korch_profile_candidate(const korch_graph* g, const korch_kernel_desc* k, int32_t warmup, int32_t reps,
                            size_t flush_bytes, void* stream, float* median_us) {
  return guard([&] {
    NEED(g);
    NEED(k);
    NEED(median_us);
    if (!g->g.finalized) fail(KORCH_E_STATE, "graph is not finalized");
    KernelDesc kd = to_desc(*k);
    std::string why;
    if (match_family(g->g, kd, &why) == KORCH_FAM_NONE) fail(KORCH_E_UNSUPPORTED, why);
    *median_us = profile_candidate(g->g, kd, std::max(0, warmup), std::max(1, reps), flush_bytes,
                                   (hipStream_t)stream);
  });
}

}  // extern "C"

// Plan compilation, code-object loading, sequential execution on one stream
// (Korch, Section 5.3) and the single-candidate profiler (Section 5.2).
#include <hip/hip_runtime_api.h>

// AMD's launch extension (declared in hip_ext.h, whose templates need the
// device compiler): a module-kernel launch whose start / stop events take the
// dispatch's own timestamps.  Work sizes are in threads (grid x block).
extern "C" hipError_t hipExtModuleLaunchKernel(hipFunction_t f, uint32_t globalWorkSizeX, uint32_t globalWorkSizeY,
                                               uint32_t globalWorkSizeZ, uint32_t localWorkSizeX,
                                               uint32_t localWorkSizeY, uint32_t localWorkSizeZ, size_t sharedMemBytes,
                                               hipStream_t hStream, void** kernelParams, void** extra,
                                               hipEvent_t startEvent, hipEvent_t stopEvent, uint32_t flags);

#include <algorithm>
#include <cstdlib>

#include "families.h"
#include "plan.h"

namespace korch {

std::vector<char> rtc_compile(const std::string& src, const std::string& name);
hipError_t launch_flush(void* p, size_t bytes, int write, hipStream_t s);
hipError_t launch_fill(void* p, size_t n, int dtype, uint64_t seed, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_touch(const void* p, size_t bytes, void* sink, hipStream_t s);
size_t touch_sink_bytes();
size_t static_scratch_bytes();
hipError_t static_scratch_setup(int dev);
void* static_scratch_address(int dev);

// Head of the static scratch reserved for hand-off counters (every plan's
// counters are a few KiB: one 128-byte line per output tile or split group).
constexpr size_t kStaticCounterBytes = (size_t)64 << 10;

#define HIPCHECK(x)                                                                             \
  do {                                                                                          \
    hipError_t e_ = (x);                                                                        \
    if (e_ != hipSuccess) fail(KORCH_E_HIP, std::string(#x) + ": " + hipGetErrorString(e_));    \
  } while (0)

void generate_plan(Plan& p) {
  if (!p.ck.empty()) return;
  std::vector<CompiledKernel> ck(p.kernels.size());
  set_kernel_prefix(p.name_prefix);
  try {
    for (size_t k = 0; k < p.kernels.size(); ++k) {
      ck[k].desc = p.kernels[k];
      ck[k].gen = generate_kernel(p.g, ck[k].desc, (int)k);
    }
  } catch (...) {
    set_kernel_prefix("korch_k");
    throw;
  }
  set_kernel_prefix("korch_k");
  p.ck = std::move(ck);
  plan_workspace(p);
}

// Kernels are compiled on the calling thread: hipRTC runs in a link namespace
// of its own with its own C library, whose per-thread state does not cover
// threads created by the process's main C library.
// Bytes of private (scratch) memory per lane that a single-kernel code object
// declares: the value of ".private_segment_fixed_size" in its AMDGPU metadata
// note (a msgpack map; the key is a 27-byte fixstr, the value a msgpack
// unsigned integer).  Registers spilled by the compiler live there.
int64_t code_scratch_bytes(const std::vector<char>& code) {
  static const std::string key = std::string(1, (char)0xbb) + ".private_segment_fixed_size";
  auto it = std::search(code.begin(), code.end(), key.begin(), key.end());
  if (it == code.end()) return 0;
  size_t i = (size_t)(it - code.begin()) + key.size();
  auto byte = [&](size_t j) -> uint64_t { return j < code.size() ? (uint8_t)code[j] : 0; };
  const uint64_t b = byte(i);
  if (b < 0x80) return (int64_t)b;
  int n = b == 0xcc ? 1 : b == 0xcd ? 2 : b == 0xce ? 4 : b == 0xcf ? 8 : 0;
  uint64_t v = 0;
  for (int j = 1; j <= n; ++j) v = v << 8 | byte(i + j);
  return (int64_t)v;
}

void compile_plan(Plan& p) {
  if (p.compiled) return;
  generate_plan(p);
  int n = (int)p.ck.size();
  bool regenerated = false;
  for (int k = 0; k < n; ++k) {
    try {
      p.ck[k].code = rtc_compile(p.ck[k].gen.source, p.ck[k].gen.name);
      // A kernel that spills registers to scratch is generated again with
      // more register relief (its family's cheaper configuration) until it
      // fits or the levels run out.
      for (int level = 1; level <= kMaxRegRelief && code_scratch_bytes(p.ck[k].code) > 0; ++level) {
        set_kernel_prefix(p.name_prefix);
        set_reg_relief(level);
        try {
          p.ck[k].gen = generate_kernel(p.g, p.ck[k].desc, k);
        } catch (...) {
          set_reg_relief(0);
          set_kernel_prefix("korch_k");
          throw;
        }
        set_reg_relief(0);
        set_kernel_prefix("korch_k");
        p.ck[k].code = rtc_compile(p.ck[k].gen.source, p.ck[k].gen.name);
        regenerated = true;
      }
    } catch (Error& e) {
      fail(e.code, "kernel " + std::to_string(k) + ": " + e.what());
    } catch (std::exception& e) {
      fail(KORCH_E_COMPILE, "kernel " + std::to_string(k) + ": " + e.what());
    }
  }
  if (regenerated) plan_workspace(p);  // a regenerated kernel may take other scratch arguments
  p.compiled = true;
}

static void unload(Plan& p) {
  for (auto& ck : p.ck) {
    if (ck.module) hipModuleUnload((hipModule_t)ck.module);
    ck.module = nullptr;
    ck.function = nullptr;
    ck.device = -1;
  }
  if (p.counters) hipFree(p.counters);
  p.counters = nullptr;
  p.loaded = false;
}

void destroy_plan_device(Plan& p) { unload(p); }

void load_plan(Plan& p) {
  compile_plan(p);
  int dev = 0;
  HIPCHECK(hipGetDevice(&dev));
  if (p.loaded && p.counter_device == dev) return;
  unload(p);
  for (auto& ck : p.ck) {
    hipModule_t m;
    HIPCHECK(hipModuleLoadData(&m, ck.code.data()));
    hipFunction_t f;
    hipError_t e = hipModuleGetFunction(&f, m, ck.gen.name.c_str());
    if (e != hipSuccess) {
      hipModuleUnload(m);
      fail(KORCH_E_HIP, "hipModuleGetFunction(" + ck.gen.name + "): " + hipGetErrorString(e));
    }
    ck.module = m;
    ck.function = f;
    ck.device = dev;
  }
  if (p.counter_bytes) {
    HIPCHECK(hipMalloc(&p.counters, p.counter_bytes));
    HIPCHECK(hipMemset(p.counters, 0, p.counter_bytes));
  }
  // set-up of allocation-free execution on this device (kept per device)
  HIPCHECK(static_scratch_setup(dev));
  p.counter_device = dev;
  p.loaded = true;
}

static bool aligned16(const void* q) { return ((uintptr_t)q & 15) == 0; }

// Launches kernels [first, first + count) of the plan (count < 0: to the end).
// starts[k] / stops[k] (arrays over all kernels of the plan, or NULL) are
// events that take the start / end timestamps of kernel k's own dispatch.
// `counters` replaces the plan's counter buffer when not NULL.
void execute_plan(Plan& p, const void* const* inputs, void* const* outputs, void* ws, size_t ws_bytes,
                  hipStream_t stream, int first, int count, void* const* starts, void* const* stops,
                  void* counters) {
  // Execution only launches: loading (code objects, the counter buffer) is
  // korch_plan_load's job, so nothing here allocates or synchronizes.
  if (!p.loaded) fail(KORCH_E_STATE, "plan is not loaded: call korch_plan_load on this device first");
  int dev = 0;
  HIPCHECK(hipGetDevice(&dev));
  if (dev != p.counter_device)
    fail(KORCH_E_STATE, "plan is loaded on device " + std::to_string(p.counter_device) + ", not on the current device " +
                            std::to_string(dev) + ": call korch_plan_load again");
  const Graph& g = p.g;
  for (size_t i = 0; i < g.inputs.size(); ++i) {
    if (!inputs || !inputs[i]) fail(KORCH_E_ARG, "input " + std::to_string(i) + " is NULL");
    if (!aligned16(inputs[i])) fail(KORCH_E_ALIGN, "input " + std::to_string(i) + " is not 16-byte aligned");
  }
  for (size_t i = 0; i < g.outputs.size(); ++i) {
    if (!outputs || !outputs[i]) fail(KORCH_E_ARG, "output " + std::to_string(i) + " is NULL");
    if (!aligned16(outputs[i])) fail(KORCH_E_ALIGN, "output " + std::to_string(i) + " is not 16-byte aligned");
  }
  if (p.ws_bytes) {
    if (!ws || ws_bytes < p.ws_bytes)
      fail(KORCH_E_WORKSPACE, "workspace needs " + std::to_string(p.ws_bytes) + " bytes");
    if (!aligned16(ws)) fail(KORCH_E_ALIGN, "workspace is not 16-byte aligned");
  }
  int nk = (int)p.ck.size();
  if (first < 0 || first > nk) fail(KORCH_E_ARG, "first kernel index out of range");
  int last = count < 0 ? nk : std::min(nk, first + count);
  char* cbase = (char*)(counters ? counters : p.counters);
  for (int k = first; k < last; ++k) {
    auto& ck = p.ck[k];
    // kernel arguments on the stack (no host allocation per launch)
    void* stack_ptr[64];
    std::vector<void*> heap_ptr;
    void** ptr = stack_ptr;
    if (ck.arg_storage.size() > 64) {
      heap_ptr.resize(ck.arg_storage.size());
      ptr = heap_ptr.data();
    }
    for (size_t a = 0; a < ck.arg_storage.size(); ++a) {
      const Storage& s = ck.arg_storage[a];
      switch (s.kind) {
        case Storage::GraphInput: ptr[a] = const_cast<void*>(inputs[s.index]); break;
        case Storage::GraphOutput: ptr[a] = outputs[s.index]; break;
        case Storage::Workspace: ptr[a] = (char*)ws + s.offset; break;
        case Storage::Counters: ptr[a] = cbase + s.offset; break;
      }
    }
    void* params[] = {(void*)ptr};
    hipEvent_t ev_start = starts ? (hipEvent_t)starts[k] : nullptr;
    hipEvent_t ev_stop = stops ? (hipEvent_t)stops[k] : nullptr;
    if (ev_start || ev_stop) {
      // the events take the timestamps of this kernel's own dispatch (no
      // separate marker packets in the stream)
      HIPCHECK(hipExtModuleLaunchKernel((hipFunction_t)ck.function, (uint32_t)(ck.gen.grid[0] * ck.gen.block[0]),
                                        (uint32_t)(ck.gen.grid[1] * ck.gen.block[1]),
                                        (uint32_t)(ck.gen.grid[2] * ck.gen.block[2]), ck.gen.block[0], ck.gen.block[1],
                                        ck.gen.block[2], 0, stream, params, nullptr, ev_start, ev_stop, 0));
      continue;
    }
    HIPCHECK(hipModuleLaunchKernel((hipFunction_t)ck.function, ck.gen.grid[0], ck.gen.grid[1], ck.gen.grid[2],
                                   ck.gen.block[0], ck.gen.block[1], ck.gen.block[2], 0, stream, params, nullptr));
  }
}

// korch_plan_execute without a workspace argument and without any allocation:
// the workspace and the hand-off counters live in the static device scratch.
// The counters this plan uses are cleared by a fill kernel first (stream
// ordered, no memset node), since the scratch keeps whatever the last call
// on this device left there.
void flush_caches(void* buf, size_t bytes, int write, hipStream_t stream) {
  HIPCHECK(launch_flush(buf, bytes, write, stream));
}

void execute_plan_noalloc(Plan& p, const void* const* inputs, void* const* outputs, hipStream_t stream) {
  if (!p.loaded) fail(KORCH_E_STATE, "plan is not loaded: call korch_plan_load on this device first");
  int dev = 0;
  HIPCHECK(hipGetDevice(&dev));
  if (dev != p.counter_device)
    fail(KORCH_E_STATE, "plan is loaded on device " + std::to_string(p.counter_device) + ", not on the current device " +
                            std::to_string(dev) + ": call korch_plan_load again");
  char* base = (char*)static_scratch_address(dev);
  if (!base) fail(KORCH_E_STATE, "static scratch not set up on this device: call korch_plan_load");
  const size_t ws_cap = static_scratch_bytes() - kStaticCounterBytes;
  if (p.counter_bytes > kStaticCounterBytes)
    fail(KORCH_E_WORKSPACE, "plan needs " + std::to_string(p.counter_bytes) + " bytes of counters; the static scratch holds " +
                                std::to_string(kStaticCounterBytes));
  if (p.ws_bytes > ws_cap)
    fail(KORCH_E_WORKSPACE, "plan needs " + std::to_string(p.ws_bytes) + " bytes of workspace; the static scratch holds " +
                                std::to_string(ws_cap) + " (use korch_plan_execute with a caller workspace)");
  if (p.counter_bytes) HIPCHECK(launch_zero(base, p.counter_bytes, stream));
  execute_plan(p, inputs, outputs, base + kStaticCounterBytes, ws_cap, stream, 0, -1, nullptr, nullptr, base);
}

// The candidate kernel as a stand-alone graph: its external tensors become
// graph inputs and its output set becomes the graph outputs.
Graph extract_subgraph(const Graph& g, const KernelDesc& kd) {
  Graph s;
  std::map<int, int> m;
  for (int u : external_inputs(g, kd)) m[u] = s.add_input(g.nodes[u].dtype, g.nodes[u].shape);
  for (int v : kd.prims) {
    const Node& n = g.nodes[v];
    std::vector<int> in;
    for (int u : n.in) in.push_back(m.at(u));
    m[v] = s.add_op(n.op, in, &n.attrs, n.dtype);
  }
  for (int o : kd.outs) s.add_output(m.at(o));
  s.finalize();
  return s;
}

void compile_candidate(const Graph& g, const KernelDesc& kd) {
  Plan p;
  p.name_prefix = "korch_cand";
  p.g = extract_subgraph(g, kd);
  KernelDesc one;
  for (size_t i = 0; i < p.g.nodes.size(); ++i)
    if (p.g.is_prim((int)i)) one.prims.push_back((int)i);
  one.outs = p.g.outputs;
  std::sort(one.outs.begin(), one.outs.end());
  p.kernels = {one};
  validate_plan(p.g, p.kernels, false);
  compile_plan(p);
}

// True when node u is computed by a kernel (not a graph input, nor a view of one).
static bool computed_in(const Graph& g, int u) {
  while (g.is_view(u)) u = g.nodes[u].in[0];
  return g.is_prim(u);
}

// With KORCH_FLUSH_WRITE=1 the flush before each timed launch writes its
// buffer instead of reading it (the caches are then full of dirty lines,
// whose write-back the timed kernel pays for).
int profile_flush_write() {
  const char* e = getenv("KORCH_FLUSH_WRITE");
  return e && e[0] == '1' ? 1 : 0;
}

// With KORCH_PROFILE_COLD=1 intermediate inputs are left cold like graph inputs.
static bool profile_warm_intermediates() {
  const char* e = getenv("KORCH_PROFILE_COLD");
  return !(e && e[0] == '1');
}

float profile_candidate(const Graph& g, const KernelDesc& kd, int warmup, int reps, size_t flush_bytes,
                        hipStream_t stream) {
  const bool warm_intermediates = profile_warm_intermediates();
  const int flush_write = profile_flush_write();
  Plan p;
  p.name_prefix = "korch_cand";
  p.g = extract_subgraph(g, kd);
  KernelDesc one;
  for (size_t i = 0; i < p.g.nodes.size(); ++i)
    if (p.g.is_prim((int)i)) one.prims.push_back((int)i);
  one.outs = p.g.outputs;
  std::sort(one.outs.begin(), one.outs.end());
  p.kernels = {one};
  validate_plan(p.g, p.kernels, false);
  compile_plan(p);
  load_plan(p);
  std::vector<void*> bufs;
  std::vector<const void*> in;
  std::vector<void*> out;
  auto alloc = [&](size_t bytes) {
    void* q = nullptr;
    HIPCHECK(hipMalloc(&q, std::max<size_t>(bytes, 256)));
    bufs.push_back(q);
    return q;
  };
  hipEvent_t* ev = nullptr;
  std::vector<float> times;
  try {
    uint64_t seed = 1;
    // The stand-alone graph's inputs are the candidate's external producers,
    // in order; those that are computed in the parent graph (not its inputs)
    // are the tensors a preceding kernel of a plan has just written.
    std::vector<int> ext = external_inputs(g, kd);
    std::vector<std::pair<const void*, size_t>> warm_bufs;
    for (size_t j = 0; j < p.g.inputs.size(); ++j) {
      const Node& n = p.g.nodes[p.g.inputs[j]];
      size_t bytes = (size_t)numel(n.shape) * dtype_bytes(n.dtype);
      void* q = alloc(bytes);
      HIPCHECK(launch_fill(q, (size_t)numel(n.shape), n.dtype, seed++, stream));
      in.push_back(q);
      if (warm_intermediates && j < ext.size() && computed_in(g, ext[j])) warm_bufs.push_back({q, bytes});
    }
    void* sink = warm_bufs.empty() ? nullptr : alloc(touch_sink_bytes());
    for (int o : p.g.outputs) {
      const Node& n = p.g.nodes[o];
      out.push_back(alloc((size_t)numel(n.shape) * dtype_bytes(n.dtype)));
    }
    void* ws = p.ws_bytes ? alloc(p.ws_bytes) : nullptr;
    void* fl = flush_bytes ? alloc(flush_bytes) : nullptr;
    for (int w = 0; w < warmup; ++w)
      execute_plan(p, in.data(), out.data(), ws, p.ws_bytes, stream, 0, -1, nullptr, nullptr, nullptr);
    ev = new hipEvent_t[2 * std::max(reps, 1)]();
    for (int r = 0; r < 2 * reps; ++r) HIPCHECK(hipEventCreate(&ev[r]));
    // Each rep: the flush (evicts L2 and the Infinity Cache), a read of every
    // intermediate input (in a plan its producer has just written it, so it
    // sits in the caches while graph inputs come from HBM), then the kernel
    // launched with a start and a stop event that take its own dispatch's
    // timestamps (no marker packets, whose serialization would add a few
    // microseconds to every candidate and bias the choice toward fewer kernels).
    for (int r = 0; r < reps; ++r) {
      if (fl) HIPCHECK(launch_flush(fl, flush_bytes, flush_write, stream));
      for (auto& b : warm_bufs) HIPCHECK(launch_touch(b.first, b.second, sink, stream));
      execute_plan(p, in.data(), out.data(), ws, p.ws_bytes, stream, 0, -1, (void* const*)&ev[2 * r],
                   (void* const*)&ev[2 * r + 1], nullptr);
    }
    HIPCHECK(hipStreamSynchronize(stream));
    for (int r = 0; r < reps; ++r) {
      float ms = 0;
      HIPCHECK(hipEventElapsedTime(&ms, ev[2 * r], ev[2 * r + 1]));
      times.push_back(ms * 1000.0f);
    }
  } catch (...) {
    hipStreamSynchronize(stream);
    if (ev) {
      for (int r = 0; r < 2 * reps; ++r) hipEventDestroy(ev[r]);
      delete[] ev;
    }
    for (void* q : bufs) hipFree(q);
    unload(p);
    throw;
  }
  for (int r = 0; r < 2 * reps; ++r) hipEventDestroy(ev[r]);
  delete[] ev;
  for (void* q : bufs) hipFree(q);
  unload(p);
  if (times.empty()) return 0.0f;
  std::sort(times.begin(), times.end());
  return times[times.size() / 2];
}

}  // namespace korch

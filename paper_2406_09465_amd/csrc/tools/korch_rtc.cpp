// Compiles one generated kernel with hipRTC in a process of its own.
//
//   korch_rtc <source file> <kernel name> <code object out> <log out> [compiler options...]
//
// The library runs it (as a child process) for every code object missing from
// its cache, so the compiler never runs inside a process that drives the GPU.
// hipRTC is loaded from the ROCm installation ($ROCM_PATH, default /opt/rocm).
// Exit status: 0 code object written; 1 compilation failed (log written);
// 2 usage, I/O or loading error (message on stderr).
#include <dlfcn.h>
#include <hip/hiprtc.h>

#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

template <class F>
static bool sym(void* h, const char* name, F& f) {
  f = reinterpret_cast<F>(dlsym(h, name));
  if (!f) std::fprintf(stderr, "korch_rtc: hipRTC lacks %s\n", name);
  return f != nullptr;
}

int main(int argc, char** argv) {
  if (argc < 5) {
    std::fprintf(stderr, "usage: korch_rtc <source> <name> <code object out> <log out> [options...]\n");
    return 2;
  }
  std::ifstream in(argv[1], std::ios::binary);
  if (!in) {
    std::fprintf(stderr, "korch_rtc: cannot read %s\n", argv[1]);
    return 2;
  }
  std::stringstream ss;
  ss << in.rdbuf();
  const std::string src = ss.str();
  const char* root = std::getenv("ROCM_PATH");
  const std::string file = std::string(root && *root ? root : "/opt/rocm") + "/lib/libhiprtc.so.7";
  void* h = dlopen(file.c_str(), RTLD_NOW | RTLD_LOCAL);
  if (!h) {
    const char* e = dlerror();
    std::fprintf(stderr, "korch_rtc: cannot load %s: %s\n", file.c_str(), e ? e : "unknown error");
    return 2;
  }
  hiprtcResult (*create)(hiprtcProgram*, const char*, const char*, int, const char**, const char**) = nullptr;
  hiprtcResult (*compile)(hiprtcProgram, int, const char**) = nullptr;
  hiprtcResult (*log_size)(hiprtcProgram, size_t*) = nullptr;
  hiprtcResult (*log)(hiprtcProgram, char*) = nullptr;
  hiprtcResult (*code_size)(hiprtcProgram, size_t*) = nullptr;
  hiprtcResult (*code)(hiprtcProgram, char*) = nullptr;
  hiprtcResult (*destroy)(hiprtcProgram*) = nullptr;
  if (!(sym(h, "hiprtcCreateProgram", create) && sym(h, "hiprtcCompileProgram", compile) &&
        sym(h, "hiprtcGetProgramLogSize", log_size) && sym(h, "hiprtcGetProgramLog", log) &&
        sym(h, "hiprtcGetCodeSize", code_size) && sym(h, "hiprtcGetCode", code) &&
        sym(h, "hiprtcDestroyProgram", destroy)))
    return 2;
  const std::string name = std::string(argv[2]) + ".hip";
  std::vector<const char*> opts(argv + 5, argv + argc);
  hiprtcProgram prog;
  if (create(&prog, src.c_str(), name.c_str(), 0, nullptr, nullptr) != HIPRTC_SUCCESS) {
    std::fprintf(stderr, "korch_rtc: hiprtcCreateProgram failed for %s\n", argv[2]);
    return 2;
  }
  if (compile(prog, (int)opts.size(), opts.data()) != HIPRTC_SUCCESS) {
    size_t ls = 0;
    log_size(prog, &ls);
    std::string text(ls, '\0');
    if (ls) log(prog, &text[0]);
    destroy(&prog);
    std::ofstream(argv[4], std::ios::binary) << text;
    return 1;
  }
  size_t cs = 0;
  code_size(prog, &cs);
  std::vector<char> obj(cs);
  code(prog, obj.data());
  destroy(&prog);
  std::ofstream out(argv[3], std::ios::binary);
  out.write(obj.data(), (std::streamsize)obj.size());
  return out ? 0 : 2;
}

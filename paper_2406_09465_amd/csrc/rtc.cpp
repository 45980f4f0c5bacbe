// Runtime compilation of generated kernels for gfx950 with hipRTC, with an
// on-disk cache of code objects keyed by a hash of source, options and the
// compiler library.
//
// hipRTC is loaded from the ROCm installation ($ROCM_PATH, default /opt/rocm)
// into a link-map namespace of its own.  hipRTC finds its compiler (comgr) by
// soname at run time; in the process's main namespace that lookup would pick
// whichever comgr another library (e.g. a framework's bundled ROCm) loaded
// first, so the generated code would depend on import order.
#include <dlfcn.h>
#include <hip/hiprtc.h>
#include <limits.h>
#include <sys/stat.h>
#include <unistd.h>
#include <utime.h>

#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <mutex>
#include <sstream>

#include "ir.h"

namespace korch {

static const char* kOptions[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                                 "-Xclang", "-packed-fp32-ops"};

namespace {

struct Rtc {
  std::string path;  // resolved file of the loaded hipRTC
  hiprtcResult (*create)(hiprtcProgram*, const char*, const char*, int, const char**, const char**) = nullptr;
  hiprtcResult (*compile)(hiprtcProgram, int, const char**) = nullptr;
  hiprtcResult (*log_size)(hiprtcProgram, size_t*) = nullptr;
  hiprtcResult (*log)(hiprtcProgram, char*) = nullptr;
  hiprtcResult (*code_size)(hiprtcProgram, size_t*) = nullptr;
  hiprtcResult (*code)(hiprtcProgram, char*) = nullptr;
  hiprtcResult (*destroy)(hiprtcProgram*) = nullptr;
  std::string error;
};

template <class F>
bool sym(void* h, const char* name, F& f, std::string& err) {
  f = reinterpret_cast<F>(dlsym(h, name));
  if (!f) err = std::string("hipRTC lacks ") + name;
  return f != nullptr;
}

const Rtc& rtc() {
  static Rtc r = [] {
    Rtc x;
    const char* root = getenv("ROCM_PATH");
    std::string file = std::string(root && *root ? root : "/opt/rocm") + "/lib/libhiprtc.so.7";
    void* h = dlmopen(LM_ID_NEWLM, file.c_str(), RTLD_NOW | RTLD_LOCAL);
    if (!h) {
      const char* e = dlerror();
      x.error = "cannot load " + file + ": " + (e ? e : "unknown error");
      return x;
    }
    char real[PATH_MAX];
    x.path = realpath(file.c_str(), real) ? real : file;
    std::string& err = x.error;
    sym(h, "hiprtcCreateProgram", x.create, err) && sym(h, "hiprtcCompileProgram", x.compile, err) &&
        sym(h, "hiprtcGetProgramLogSize", x.log_size, err) && sym(h, "hiprtcGetProgramLog", x.log, err) &&
        sym(h, "hiprtcGetCodeSize", x.code_size, err) && sym(h, "hiprtcGetCode", x.code, err) &&
        sym(h, "hiprtcDestroyProgram", x.destroy, err);
    return x;
  }();
  return r;
}

std::atomic<unsigned> tmp_counter{0};

}  // namespace

static uint64_t fnv1a(const std::string& s, uint64_t h = 1469598103934665603ULL) {
  for (unsigned char c : s) {
    h ^= c;
    h *= 1099511628211ULL;
  }
  return h;
}

static std::string cache_dir() {
  const char* d = getenv("KORCH_CACHE_DIR");
  if (d && *d) return d;
  const char* home = getenv("HOME");
  return std::string(home ? home : "/tmp") + "/.cache/korch";
}

static void mkdirs(const std::string& path) {
  std::string cur;
  std::stringstream ss(path);
  std::string part;
  if (!path.empty() && path[0] == '/') cur = "/";
  while (std::getline(ss, part, '/')) {
    if (part.empty()) continue;
    cur += part + "/";
    mkdir(cur.c_str(), 0755);
  }
}

std::vector<char> rtc_compile(const std::string& src, const std::string& name) {
  std::string opts;
  for (auto o : kOptions) opts += std::string(o) + " ";
  const Rtc& R = rtc();
  if (!R.error.empty()) fail(KORCH_E_COMPILE, R.error);
  uint64_t h = fnv1a(src, fnv1a(opts + R.path + name));
  char hex[32];
  snprintf(hex, sizeof(hex), "%016llx", (unsigned long long)h);
  std::string dir = cache_dir();
  std::string path = dir + "/" + name + "_" + hex + ".co";
  {
    std::ifstream f(path, std::ios::binary);
    if (f) {
      std::vector<char> code((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
      if (!code.empty()) {
        utime(path.c_str(), nullptr);  // mark as recently used (cache pruning keeps it)
        return code;
      }
    }
  }
  // hipRTC's in-process compiler keeps process-global state (LLVM's option
  // parsing among it) and is not safe to call from several threads at once;
  // callers that compile from several threads take turns here.
  static std::mutex compile_mutex;
  std::lock_guard<std::mutex> lock(compile_mutex);
  hiprtcProgram prog;
  if (R.create(&prog, src.c_str(), (name + ".hip").c_str(), 0, nullptr, nullptr) != HIPRTC_SUCCESS)
    fail(KORCH_E_COMPILE, "hiprtcCreateProgram failed for " + name);
  hiprtcResult r = R.compile(prog, (int)(sizeof(kOptions) / sizeof(kOptions[0])), kOptions);
  if (r != HIPRTC_SUCCESS) {
    size_t ls = 0;
    R.log_size(prog, &ls);
    std::string log(ls, '\0');
    if (ls) R.log(prog, &log[0]);
    R.destroy(&prog);
    if (log.size() > 4000) log = log.substr(0, 4000);
    fail(KORCH_E_COMPILE, "hipRTC failed for " + name + ": " + log);
  }
  size_t cs = 0;
  R.code_size(prog, &cs);
  std::vector<char> code(cs);
  R.code(prog, code.data());
  R.destroy(&prog);
  mkdirs(dir);
  std::string tmp = path + ".tmp" + std::to_string(getpid()) + "." + std::to_string(tmp_counter++);
  {
    std::ofstream f(tmp, std::ios::binary);
    f.write(code.data(), (std::streamsize)code.size());
  }
  rename(tmp.c_str(), path.c_str());
  return code;
}

}  // namespace korch

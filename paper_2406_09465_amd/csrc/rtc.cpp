// Runtime compilation of generated kernels for gfx950 with hipRTC, with an
// on-disk cache of code objects keyed by a hash of source and options.
#include <hip/hiprtc.h>
#include <sys/stat.h>
#include <unistd.h>
#include <utime.h>

#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <mutex>
#include <sstream>

#include "ir.h"

namespace korch {

static const char* kOptions[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                                 "-Xclang", "-packed-fp32-ops"};

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
  int ver = 0;
  {
    int major = 0, minor = 0;
    hiprtcVersion(&major, &minor);
    ver = major * 1000 + minor;
  }
  uint64_t h = fnv1a(src, fnv1a(opts + std::to_string(ver) + name));
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
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src.c_str(), (name + ".hip").c_str(), 0, nullptr, nullptr) != HIPRTC_SUCCESS)
    fail(KORCH_E_COMPILE, "hiprtcCreateProgram failed for " + name);
  hiprtcResult r = hiprtcCompileProgram(prog, (int)(sizeof(kOptions) / sizeof(kOptions[0])), kOptions);
  if (r != HIPRTC_SUCCESS) {
    size_t ls = 0;
    hiprtcGetProgramLogSize(prog, &ls);
    std::string log(ls, '\0');
    if (ls) hiprtcGetProgramLog(prog, &log[0]);
    hiprtcDestroyProgram(&prog);
    if (log.size() > 4000) log = log.substr(0, 4000);
    fail(KORCH_E_COMPILE, "hipRTC failed for " + name + ": " + log);
  }
  size_t cs = 0;
  hiprtcGetCodeSize(prog, &cs);
  std::vector<char> code(cs);
  hiprtcGetCode(prog, code.data());
  hiprtcDestroyProgram(&prog);
  mkdirs(dir);
  std::string tmp = path + ".tmp" + std::to_string(getpid());
  {
    std::ofstream f(tmp, std::ios::binary);
    f.write(code.data(), (std::streamsize)code.size());
  }
  rename(tmp.c_str(), path.c_str());
  return code;
}

}  // namespace korch

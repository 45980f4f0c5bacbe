// Runtime compilation of generated kernels for gfx950 with hipRTC, with an
// on-disk cache of code objects keyed by a hash of source, options and the
// compiler library.
//
// A code object missing from the cache is compiled by the helper executable
// `korch_rtc` (built next to this library) in a child process: hipRTC's
// in-process compiler keeps process-global state and brings its own copy of
// the compiler libraries, and running it inside a process that also drives
// the GPU (and whose framework may have loaded another compiler library) is
// avoided altogether.  The helper loads hipRTC from the ROCm installation
// ($ROCM_PATH, default /opt/rocm).
#include <dlfcn.h>
#include <limits.h>
#include <spawn.h>
#include <sys/stat.h>
#include <sys/wait.h>
#include <unistd.h>
#include <utime.h>

#include <atomic>
#include <cerrno>
#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <mutex>
#include <sstream>

#include "ir.h"

extern char** environ;

namespace korch {

static const char* kOptions[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                                 "-Xclang", "-packed-fp32-ops"};

namespace {

// The hipRTC library the helper loads (its resolved path is part of the cache key).
const std::string& hiprtc_path() {
  static const std::string p = [] {
    const char* root = getenv("ROCM_PATH");
    std::string file = std::string(root && *root ? root : "/opt/rocm") + "/lib/libhiprtc.so.7";
    char real[PATH_MAX];
    return std::string(realpath(file.c_str(), real) ? real : file.c_str());
  }();
  return p;
}

// The helper executable: korch_rtc in the directory of this library.
const std::string& helper_path() {
  static const std::string p = [] {
    Dl_info info;
    std::string dir = ".";
    if (dladdr((void*)&hiprtc_path, &info) && info.dli_fname) {
      std::string f = info.dli_fname;
      size_t slash = f.rfind('/');
      if (slash != std::string::npos) dir = f.substr(0, slash);
    }
    return dir + "/korch_rtc";
  }();
  return p;
}

std::atomic<unsigned> tmp_counter{0};

std::string read_file(const std::string& path) {
  std::ifstream f(path, std::ios::binary);
  std::stringstream ss;
  ss << f.rdbuf();
  return ss.str();
}

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
  uint64_t h = fnv1a(src, fnv1a(opts + hiprtc_path() + name));
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
  mkdirs(dir);
  const std::string tmp = path + ".tmp" + std::to_string(getpid()) + "." + std::to_string(tmp_counter++);
  const std::string src_file = tmp + ".hip", obj_file = tmp + ".co", log_file = tmp + ".log";
  {
    std::ofstream f(src_file, std::ios::binary);
    f.write(src.data(), (std::streamsize)src.size());
    if (!f) fail(KORCH_E_COMPILE, "cannot write " + src_file);
  }
  std::vector<std::string> args = {helper_path(), src_file, name, obj_file, log_file};
  for (auto o : kOptions) args.push_back(o);
  std::vector<char*> argv;
  for (auto& a : args) argv.push_back(&a[0]);
  argv.push_back(nullptr);
  pid_t pid;
  int rc = posix_spawn(&pid, helper_path().c_str(), nullptr, nullptr, argv.data(), environ);
  int status = 0;
  if (rc == 0) {
    while (waitpid(pid, &status, 0) < 0 && errno == EINTR) {
    }
  }
  std::string log = read_file(log_file);
  std::vector<char> code;
  if (rc == 0 && WIFEXITED(status) && WEXITSTATUS(status) == 0) {
    std::string obj = read_file(obj_file);
    code.assign(obj.begin(), obj.end());
  }
  unlink(src_file.c_str());
  unlink(log_file.c_str());
  if (code.empty()) {
    unlink(obj_file.c_str());
    if (rc != 0) fail(KORCH_E_COMPILE, "cannot run " + helper_path() + " (build the library)");
    if (log.size() > 4000) log = log.substr(0, 4000);
    fail(KORCH_E_COMPILE, "hipRTC failed for " + name + ": " +
                              (log.empty() ? "helper exited with status " + std::to_string(status) : log));
  }
  rename(obj_file.c_str(), path.c_str());
  return code;
}

}  // namespace korch

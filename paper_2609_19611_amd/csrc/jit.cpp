// Run-time specialisation of the per-location kernels (see jit.h).
#include "jit.h"

#include <dlfcn.h>
#include <fcntl.h>
#include <poll.h>
#include <pthread.h>
#include <signal.h>
#include <spawn.h>
#include <sys/wait.h>
#include <unistd.h>

#include <cerrno>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <sstream>

extern char** environ;

namespace dg {

namespace {

std::mutex g_mu;
// Loaded modules: (device, source) -> module and the number of holders.
struct Loaded {
  hipModule_t mod = nullptr;
  int refs = 0;
};
std::map<std::pair<int, std::string>, Loaded> g_modules;
// Compiled code objects by source, with a use stamp; at most kCodeCache are
// kept (least recently used dropped first).
struct Code {
  std::vector<char> bytes;
  uint64_t stamp = 0;
};
const size_t kCodeCache = 128;
std::map<std::string, Code> g_code;
uint64_t g_clock = 0;

void remember_code(const std::string& source, const std::vector<char>& code) {  // g_mu held
  Code& c = g_code[source];
  c.bytes = code;
  c.stamp = ++g_clock;
  while (g_code.size() > kCodeCache) {
    auto oldest = g_code.begin();
    for (auto it = g_code.begin(); it != g_code.end(); ++it)
      if (it->second.stamp < oldest->second.stamp) oldest = it;
    g_code.erase(oldest);
  }
}

// The compile helper program beside this library (dirigo_jitc), or empty.
std::string helper_path() {
  Dl_info info;
  if (!dladdr(reinterpret_cast<void*>(&helper_path), &info) || !info.dli_fname) return std::string();
  std::string p(info.dli_fname);
  const size_t slash = p.rfind('/');
  p = (slash == std::string::npos ? std::string(".") : p.substr(0, slash)) + "/dirigo_jitc";
  return access(p.c_str(), X_OK) == 0 ? p : std::string();
}

// Compiles `src` in a child process running the helper: the source goes to
// its stdin, a status byte and the code object (or the log) come back on
// its stdout.  The child is a separate program image that never touches
// the GPU; the caller's process only waits for it (at most kHelperSeconds).
// The pipes are close-on-exec, so a child started by another thread never
// holds this call's pipe ends; a child that exits early cannot raise
// SIGPIPE in the caller (blocked during the write, then consumed).
const int kHelperSeconds = 900;

bool compile_in_helper(const std::string& helper, const std::string& src, std::vector<char>* code,
                       std::string* log) {
  int in[2], out[2];
  if (pipe2(in, O_CLOEXEC) != 0) {
    *log = "pipe failed";
    return false;
  }
  if (pipe2(out, O_CLOEXEC) != 0) {
    close(in[0]);
    close(in[1]);
    *log = "pipe failed";
    return false;
  }
  posix_spawn_file_actions_t fa;
  posix_spawn_file_actions_init(&fa);
  posix_spawn_file_actions_adddup2(&fa, in[0], 0);  // (dup2 leaves the copies inheritable)
  posix_spawn_file_actions_adddup2(&fa, out[1], 1);
  char* const argv[] = {const_cast<char*>(helper.c_str()), nullptr};
  pid_t pid = -1;
  const int rc = posix_spawn(&pid, helper.c_str(), &fa, nullptr, argv, environ);
  posix_spawn_file_actions_destroy(&fa);
  close(in[0]);
  close(out[1]);
  if (rc != 0) {
    close(in[1]);
    close(out[0]);
    *log = "cannot start " + helper;
    return false;
  }
  // (The helper reads its whole input before it writes anything.)
  sigset_t pipe_set, old_set;
  sigemptyset(&pipe_set);
  sigaddset(&pipe_set, SIGPIPE);
  pthread_sigmask(SIG_BLOCK, &pipe_set, &old_set);
  size_t done = 0;
  bool broken = false;
  while (done < src.size()) {
    const ssize_t w = write(in[1], src.data() + done, src.size() - done);
    if (w < 0 && errno == EINTR) continue;
    if (w <= 0) {
      broken = w < 0 && errno == EPIPE;
      break;
    }
    done += (size_t)w;
  }
  close(in[1]);
  if (broken) {
    const struct timespec zero = {0, 0};
    while (sigtimedwait(&pipe_set, nullptr, &zero) < 0 && errno == EINTR) {
    }
  }
  pthread_sigmask(SIG_SETMASK, &old_set, nullptr);
  std::vector<char> buf;
  char chunk[1 << 16];
  bool timed_out = false;
  for (;;) {
    struct pollfd pf = {out[0], POLLIN, 0};
    const int pr = poll(&pf, 1, kHelperSeconds * 1000);
    if (pr < 0 && errno == EINTR) continue;
    if (pr == 0) {
      timed_out = true;
      kill(pid, SIGKILL);
      break;
    }
    const ssize_t r = read(out[0], chunk, sizeof chunk);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) break;
    buf.insert(buf.end(), chunk, chunk + r);
  }
  close(out[0]);
  int status = 0;
  while (waitpid(pid, &status, 0) < 0 && errno == EINTR) {
  }
  const bool ok = !timed_out && done == src.size() && WIFEXITED(status) && WEXITSTATUS(status) == 0 &&
                  !buf.empty() && buf[0] == 0;
  if (!ok) {
    *log = timed_out ? std::string("compile helper timed out")
                     : buf.size() > 1 ? std::string(buf.begin() + 1, buf.end()) : std::string("compile helper failed");
    return false;
  }
  code->assign(buf.begin() + 1, buf.end());
  return !code->empty();
}

// A process that uses PyTorch has its bundled HIP runtime loaded, and with
// it an older runtime compiler that generates markedly slower code for these
// kernels; the helper always compiles with the ROCm installation's.  Without
// the helper (or with DIRIGO_JIT_INPROC=1) the kernels are compiled in
// process.
bool compile(const std::string& src, std::vector<char>* code, std::string* log) {
  const char* e = std::getenv("DIRIGO_JIT_INPROC");
  if (!(e && std::strcmp(e, "1") == 0)) {
    static const std::string helper = helper_path();
    if (!helper.empty()) return compile_in_helper(helper, src, code, log);
  }
  return jit_compile_source(src, code, log);
}

}  // namespace

bool jit_enabled() {
  const char* e = std::getenv("DIRIGO_JIT");
  return !(e && std::strcmp(e, "0") == 0);
}

bool jit_load(const std::string& source, JitModule* out, std::string* log) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *log = "hipGetDevice failed";
    return false;
  }
  std::vector<char> code;
  out->mod = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    auto mit = g_modules.find({dev, source});
    if (mit != g_modules.end()) {
      ++mit->second.refs;
      out->mod = mit->second.mod;
    } else {
      auto it = g_code.find(source);
      if (it != g_code.end()) {
        code = it->second.bytes;
        it->second.stamp = ++g_clock;
      }
    }
  }
  if (!out->mod) {
    if (code.empty()) {
      if (!compile(source, &code, log)) return false;
      std::lock_guard<std::mutex> lock(g_mu);
      remember_code(source, code);
    }
    hipModule_t m = nullptr;
    hipError_t e = hipModuleLoadData(&m, code.data());
    if (e != hipSuccess) {
      *log = std::string("hipModuleLoadData: ") + hipGetErrorString(e);
      return false;
    }
    std::lock_guard<std::mutex> lock(g_mu);
    Loaded& L = g_modules[{dev, source}];
    if (L.mod) {
      (void)hipModuleUnload(m);  // another thread loaded it meanwhile
    } else {
      L.mod = m;
    }
    ++L.refs;
    out->mod = L.mod;
  }
  out->dev = dev;
  out->source = source;
  // A module holds the enumeration kernels, the comparison kernel or the
  // DAG kernels;
  // a name it lacks leaves a null function.  The failed lookup also sets
  // the thread's last HIP error, which is cleared here so that it is not
  // reported by the next launch check.
  auto get = [&](const char* name, hipFunction_t* f) {
    if (hipModuleGetFunction(f, out->mod, name) != hipSuccess) {
      *f = nullptr;
      (void)hipGetLastError();
    }
  };
  get("dg_sizes", &out->sizes);
  get("dg_fill", &out->fill);
  get("dg_enumerate", &out->enumerate);
  get("dg_compare", &out->compare);
  get("dg_enumerate_wide", &out->enumerate_wide);
  get("dg_dag_sizes", &out->dag_sizes);
  get("dg_dag_fill", &out->dag_fill);
  get("dg_dag_onepass", &out->dag_onepass);
  return true;
}

void jit_release(JitModule* m) {
  if (!m || !m->mod) return;
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_modules.find({m->dev, m->source});
  if (it != g_modules.end() && --it->second.refs == 0) {
    int cur = -1;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (hipSetDevice(m->dev) == hipSuccess) (void)hipModuleUnload(it->second.mod);
    if (have) (void)hipSetDevice(cur);
    g_modules.erase(it);
  }
  *m = JitModule{};
}

}  // namespace dg

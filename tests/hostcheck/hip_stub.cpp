// A stand-in HIP runtime for the host-only build of libckpt (every source
// compiled with --offload-host-only under AddressSanitizer and UBSan): kernel
// launches are recorded and checked instead of run.
//
// Device memory is never real here: the driver hands the library fake device
// addresses from hc_alloc (a range no host mapping uses), so any host
// dereference of device memory faults at once.  Every launch's pointer
// arguments must lie inside one of those allocations (or the library's static
// scratch); the bf16 GEMM's argument block is checked over the whole extent
// each operand spans for the launch's shape, leading dimensions, operand forms,
// gathers, epilogue and split count.  Grid and block sizes are checked
// against the device limits.  Errors are counted and the first few printed.
#include <cxxabi.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../paper_1604_06174_amd/csrc/gemm_bf16_kernel.h"
#include "../../paper_1604_06174_amd/csrc/kernel_args.h"

namespace {

constexpr uintptr_t kFakeBase = uintptr_t(0x7a0000000000ull);
constexpr uintptr_t kFakeEnd = uintptr_t(0x7b0000000000ull);

struct Region {
  uintptr_t lo, hi;
  std::string name;
};

struct Param {
  enum Kind { PTR, SCALAR, GEMM_BF16, CONV, WGRAD, GEMM_F32 } kind;
};

struct KernelInfo {
  std::string mangled, pretty;
  std::vector<Param> params;
  std::vector<std::string> targs;  // template arguments
  bool parsed = false;
  uint64_t launches = 0;
};

struct Config {
  dim3 grid, block;
  size_t shm;
  hipStream_t s;
};

// All state lives in one function-local object: the other objects' static
// constructors register their kernels before any namespace-scope object of
// this file would be constructed.
struct State {
  std::mutex mu;
  std::map<const void *, KernelInfo> kernels;  // host stub -> kernel
  std::map<const void *, Region> vars;         // host shadow of a __device__ variable
  std::vector<Region> regions;
  std::vector<Config> cfg;
  uintptr_t next = kFakeBase;
  uint64_t launches = 0, errors = 0, ptr_checks = 0, extent_checks = 0;
  hipError_t last = hipSuccess;
};

State &S() {
  static State *s = new State;  // never destroyed: unregistration may run after exit handlers
  return *s;
}

void error(const std::string &msg) {
  ++S().errors;
  if (S().errors <= 20) fprintf(stderr, "hostcheck: %s\n", msg.c_str());
}

const Region *find(uintptr_t p) {
  for (const Region &r : S().regions)
    if (p >= r.lo && p < r.hi) return &r;
  return nullptr;
}

std::string hex(uintptr_t p) {
  char b[32];
  snprintf(b, sizeof b, "0x%llx", (unsigned long long)p);
  return b;
}

// a device pointer argument: null, or inside a caller allocation
void check_ptr(const KernelInfo &k, const char *what, const void *p) {
  ++S().ptr_checks;
  if (!p) return;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  if (!find(a)) error(k.pretty + ": " + what + " = " + hex(a) + " is in no device allocation");
}

// [p, p + bytes) wholly inside one allocation
void check_extent(const KernelInfo &k, const char *what, const void *p, uint64_t bytes) {
  ++S().extent_checks;
  if (!p) {
    error(k.pretty + ": " + what + " is null");
    return;
  }
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  const Region *r = find(a);
  if (!r) {
    error(k.pretty + ": " + what + " = " + hex(a) + " is in no device allocation");
    return;
  }
  if (bytes > r->hi - a)
    error(k.pretty + ": " + what + " spans " + std::to_string(bytes) + " bytes from offset " +
          std::to_string(a - r->lo) + " of " + r->name + " (" + std::to_string(r->hi - r->lo) +
          " bytes)");
}

// top-level comma split of s[b, e)
std::vector<std::string> split_top(const std::string &s, size_t b, size_t e) {
  std::vector<std::string> out;
  int depth = 0;
  size_t start = b;
  for (size_t i = b; i < e; ++i) {
    const char c = s[i];
    if (c == '<' || c == '(' || c == '[') ++depth;
    if (c == '>' || c == ')' || c == ']') --depth;
    if (c == ',' && depth == 0) {
      out.push_back(s.substr(start, i - start));
      start = i + 1;
    }
  }
  if (e > start) out.push_back(s.substr(start, e - start));
  for (std::string &t : out) {
    while (!t.empty() && t.front() == ' ') t.erase(t.begin());
    while (!t.empty() && t.back() == ' ') t.pop_back();
  }
  return out;
}

void parse(KernelInfo &k) {
  k.parsed = true;
  // this demangler predates the DF16b code of __bf16: stand in another
  // builtin (Dh, "half"; like DF16b not a substitution candidate, so the
  // back-references keep their indices) and name it __bf16 again after
  std::string m = k.mangled;
  for (size_t at; (at = m.find("DF16b")) != std::string::npos;) m.replace(at, 5, "Dh");
  int st = 0;
  char *d = abi::__cxa_demangle(m.c_str(), nullptr, nullptr, &st);
  k.pretty = (st == 0 && d) ? d : k.mangled;
  free(d);
  for (size_t at; (at = k.pretty.find("half")) != std::string::npos;) k.pretty.replace(at, 4, "__bf16");
  const std::string &p = k.pretty;
  // parameter list: the last top-level "( ... )"
  if (p.empty() || p.back() != ')') {
    error("cannot parse kernel signature: " + p);
    return;
  }
  int depth = 0;
  size_t open = std::string::npos;
  for (size_t i = p.size(); i-- > 0;) {
    if (p[i] == ')') ++depth;
    if (p[i] == '(' && --depth == 0) {
      open = i;
      break;
    }
  }
  if (open == std::string::npos) {
    error("cannot parse kernel signature: " + p);
    return;
  }
  // template arguments: the "<...>" right before the parameter list
  if (open > 0 && p[open - 1] == '>') {
    int dd = 0;
    for (size_t i = open; i-- > 0;) {
      if (p[i] == '>') ++dd;
      if (p[i] == '<' && --dd == 0) {
        k.targs = split_top(p, i + 1, open - 1);
        break;
      }
    }
  }
  for (const std::string &t : split_top(p, open + 1, p.size() - 1)) {
    Param q;
    if (t.empty() || t == "void") continue;
    if (t.back() == '*') q.kind = Param::PTR;
    else if (t == "ckpt::gb::Args") q.kind = Param::GEMM_BF16;
    else if (t == "ckpt::ConvArgs") q.kind = Param::CONV;
    else if (t == "ckpt::WgArgs") q.kind = Param::WGRAD;
    else if (t == "ckpt::GemmArgs") q.kind = Param::GEMM_F32;
    else if (t == "int" || t == "long" || t == "unsigned int" || t == "unsigned long" || t == "float" ||
             t == "double" || t == "bool" || t == "long long" || t == "unsigned long long")
      q.kind = Param::SCALAR;
    else {
      error(p + ": parameter type '" + t + "' unknown to the launch checker");
      q.kind = Param::SCALAR;
    }
    k.params.push_back(q);
  }
}

uint64_t rows_span(uint64_t rows, uint64_t ld, uint64_t cols) { return rows ? (rows - 1) * ld + cols : 0; }

// HC_GEMM_LOG=<file>: one line per bf16 GEMM launch (mangled name, grid,
// M, N, K, k per split, epilogue, A and B forms, gather geometry, whether the
// epilogue also writes the batch-norm output and reads a shortcut, and the
// products of a batch), for attaching shapes to a profiler's per-dispatch
// records
void log_gemm(const KernelInfo &k, const ckpt::gb::Args &a, dim3 grid, int epi, int ga, int gb) {
  static FILE *f = [] {
    const char *p = std::getenv("HC_GEMM_LOG");
    return p ? std::fopen(p, "w") : nullptr;
  }();
  if (!f) return;
  std::fprintf(f, "%s %u %u %u %d %d %d %d %d %d %d %d %d %d %d %d %d %d %d %d %d %d\n", k.mangled.c_str(),
               grid.x, grid.y, grid.z, a.M, a.N, a.K, a.kper, epi, ga, gb, a.H, a.W, a.Ho, a.Wo, a.R, a.S,
               a.cshift, a.lda, a.Rb != nullptr, a.Xr != nullptr, a.nbatch);
  std::fflush(f);
}

// the whole extent of every operand of a bf16 GEMM launch
void check_gemm_bf16(const KernelInfo &k, const ckpt::gb::Args &a, dim3 grid) {
  using namespace ckpt::gb;
  if (k.targs.size() != 12) {
    error(k.pretty + ": unexpected template arguments");
    return;
  }
  const bool AK = k.targs[4] == "true", BK = k.targs[5] == "true";
  const uint64_t ta = k.targs[6] == "float" ? 4 : 2;
  const int EPI = std::atoi(k.targs[7].c_str()), GA = std::atoi(k.targs[8].c_str()),
            GB = std::atoi(k.targs[9].c_str());
  const int BM = std::atoi(k.targs[0].c_str()), BN = std::atoi(k.targs[1].c_str());
  log_gemm(k, a, grid, EPI, GA, GB);
  const uint64_t M = uint64_t(a.M), N = uint64_t(a.N), K = uint64_t(a.K);
  if (a.M <= 0 || a.N <= 0 || a.K < 0) error(k.pretty + ": non-positive M or N");
  if (grid.x != (N + BN - 1) / BN || grid.y != (M + BM - 1) / BM)
    error(k.pretty + ": grid does not cover the product's tiles exactly");
  // a batch of products: grid.z = the products, each over the whole k range
  const uint64_t nb = a.nbatch > 0 ? uint64_t(a.nbatch) : 1;
  if (a.nbatch > 0 && (grid.z != nb || uint64_t(a.kper) < K))
    error(k.pretty + ": a batch takes one workgroup layer per product and one k split");
  if (a.nbatch == 0 && (a.kper <= 0 || uint64_t(a.kper) * grid.z < K))
    error(k.pretty + ": k splits do not cover K");
  const uint64_t ba = (nb - 1) * uint64_t(a.bstrA), bc = (nb - 1) * uint64_t(a.bstrC),
                 br = (nb - 1) * uint64_t(a.bstrR);
  const uint64_t C = a.cshift >= 0 ? uint64_t(1) << a.cshift : 0;
  // A
  if (GA == G_DENSE) {
    check_extent(k, "A", a.A, (ba + (AK ? rows_span(M, a.lda, K) : rows_span(K, a.lda, M))) * ta);
  } else if (GA == GA_FWD || GA == GA_FWDT) {
    const uint64_t pix = uint64_t(a.Ho) * a.Wo;
    if (M % pix) error(k.pretty + ": forward gather rows are not whole images");
    check_extent(k, "A (gathered input)", a.A, (M / pix) * a.H * a.W * C * 2);
  } else if (GA == GA_DGRAD || GA == GA_DGRADT) {
    const uint64_t pix = uint64_t(a.H) * a.W;
    if (M % pix) error(k.pretty + ": data-gradient gather rows are not whole images");
    check_extent(k, "A (gathered output gradient)", a.A, (M / pix) * a.Ho * a.Wo * C * 2);
  } else if (GA == GA_CAT) {
    check_extent(k, "A (first part)", a.A, rows_span(M, a.lda, a.K1) * 2);
    check_extent(k, "A2 (second part)", a.A2, rows_span(M, a.lda2, K - a.K1) * 2);
  } else {
    error(k.pretty + ": unknown A form");
  }
  // the tap-uniform gathers leave out the per-chunk k bound and keep one bit per tap
  if ((GA == GA_FWDT || GA == GA_DGRADT) &&
      (a.cshift < 0 || (1 << a.cshift) % KS || a.K % KS || a.kper % KS || a.R * a.R > 32 || (GA == GA_DGRADT && a.S != 1) ||
       a.nbatch > 0))
    error(k.pretty + ": tap-uniform gather outside its conditions");
  // B
  if (GB == G_DENSE) {
    check_extent(k, "B", a.B, (BK ? rows_span(N, a.ldb, K) : rows_span(K, a.ldb, N)) * 2);
  } else if (GB == GB_WGRAD) {
    const uint64_t pix = uint64_t(a.Ho) * a.Wo;
    if (K % pix) error(k.pretty + ": weight-gradient pixels are not whole images");
    check_extent(k, "B (gathered input)", a.B, (K / pix) * a.H * a.W * C * 2);
  } else if (GB == GB_WDGRAD) {
    check_extent(k, "B (forward weights)", a.B, C * a.R * a.R * N * 2);
  } else {
    error(k.pretty + ": unknown B form");
  }
  if (a.Rb && EPI != ckpt::GEMM_EPI_BF16STATS) error(k.pretty + ": a batch-norm apply output without BF16STATS");
  // result and epilogue operands
  const uint64_t cz = a.nbatch > 0 ? 1 : uint64_t(grid.z);
  if (EPI == ckpt::GEMM_EPI_BF16STATS) {
    check_extent(k, "Cb", a.Cb, rows_span(M, a.ldc, N) * 2);
    if (a.stats) check_extent(k, "stats", a.stats, uint64_t(grid.y) * 2 * N * 8);
    if (a.Rb) {  // the batch-norm apply output of a re-run
      check_extent(k, "Rb", a.Rb, rows_span(M, a.ldc, N) * 2);
      if (a.Xr) check_extent(k, "Xr (residual)", a.Xr, rows_span(M, a.ldc, N) * 2);
      check_extent(k, "apply statistics", a.ast, 2 * N * 4);
      check_extent(k, "apply gamma", a.ag, N * 4);
      check_extent(k, "apply beta", a.ab, N * 4);
    }
  } else {
    check_extent(k, "C", a.C, (bc + (cz - 1) * M * a.ldc + rows_span(M, a.ldc, N)) * 4);
  }
  if (EPI == ckpt::GEMM_EPI_ADD || EPI == ckpt::GEMM_EPI_ADDMASK)
    check_extent(k, "D", a.D, rows_span(M, a.ldd, N) * 4);
  if (EPI == ckpt::GEMM_EPI_ADDMASK) check_extent(k, "mask", a.Ym, rows_span(M, a.ldd, N) * 2);
  if (EPI == ckpt::GEMM_EPI_BNBWD) {
    check_extent(k, "mask", a.Ym, rows_span(M, a.ldc, N) * 2);
    check_extent(k, "batch-norm input", a.Cv, rows_span(M, a.ldc, N) * 2);
    check_extent(k, "batch-norm statistics", a.bst, 2 * N * 4);
    check_extent(k, "backward partial sums", a.stats, uint64_t(grid.y) * 2 * N * 8);
  }
  if (EPI == ckpt::GEMM_EPI_ROWSOFTMAX) {
    check_extent(k, "bias", a.bias, N * 4);
    check_extent(k, "row statistics", a.rstat, (br + M * grid.x * 2) * 4);
  } else if (EPI == ckpt::GEMM_EPI_STORE && a.bias) {
    check_extent(k, "bias", a.bias, N * 4);
  }
}

void check_launch(const void *f, dim3 grid, dim3 block, void **args, size_t shm) {
  std::lock_guard<std::mutex> lock(S().mu);
  ++S().launches;
  auto it = S().kernels.find(f);
  if (it == S().kernels.end()) {
    error("launch of an unregistered kernel");
    S().last = hipErrorInvalidDeviceFunction;
    return;
  }
  KernelInfo &k = it->second;
  if (!k.parsed) parse(k);
  ++k.launches;
  if (grid.x == 0 || grid.y == 0 || grid.z == 0 || grid.y > 65535 || grid.z > 65535 ||
      grid.x > 0x7fffffffu)
    error(k.pretty + ": grid " + std::to_string(grid.x) + "x" + std::to_string(grid.y) + "x" +
          std::to_string(grid.z) + " outside the device limits");
  const uint64_t threads = uint64_t(block.x) * block.y * block.z;
  if (threads == 0 || threads > 1024) error(k.pretty + ": block of " + std::to_string(threads) + " threads");
  if (shm > 160 * 1024) error(k.pretty + ": " + std::to_string(shm) + " bytes of dynamic LDS");
  for (size_t i = 0; i < k.params.size(); ++i) {
    switch (k.params[i].kind) {
      case Param::PTR: check_ptr(k, ("argument " + std::to_string(i)).c_str(), *static_cast<void **>(args[i])); break;
      case Param::GEMM_BF16: check_gemm_bf16(k, *static_cast<const ckpt::gb::Args *>(args[i]), grid); break;
      case Param::CONV: {
        const ckpt::ConvArgs &c = *static_cast<const ckpt::ConvArgs *>(args[i]);
        const void *ps[] = {c.X, c.Wt, c.Y, c.E0, c.E1, c.stats, c.tst, c.tg, c.tb, c.rout};
        for (const void *q : ps) check_ptr(k, "ConvArgs field", q);
        break;
      }
      case Param::WGRAD: {
        const ckpt::WgArgs &w = *static_cast<const ckpt::WgArgs *>(args[i]);
        const void *ps[] = {w.X, w.DY, w.part, w.tst, w.tg, w.tb};
        for (const void *q : ps) check_ptr(k, "WgArgs field", q);
        break;
      }
      case Param::GEMM_F32: {
        const ckpt::GemmArgs &g = *static_cast<const ckpt::GemmArgs *>(args[i]);
        const void *ps[] = {g.A, g.B, g.C, g.D, g.bias, g.Z};
        for (const void *q : ps) check_ptr(k, "GemmArgs field", q);
        break;
      }
      case Param::SCALAR: break;
    }
  }
}

}  // namespace

// ---- the driver's controls -------------------------------------------------
extern "C" {

// a fake device allocation of `bytes` (256-byte aligned, 64 KiB apart)
uintptr_t hc_alloc(uint64_t bytes, const char *name) {
  std::lock_guard<std::mutex> lock(S().mu);
  const uintptr_t p = S().next;
  S().next += (bytes + 65535) / 65536 * 65536 + 65536;
  if (S().next >= kFakeEnd) {
    error("fake device address space exhausted");
    return 0;
  }
  S().regions.push_back({p, p + bytes, name ? name : "?"});
  return p;
}

// drop every caller allocation (the static scratch stays)
void hc_free_all(void) {
  std::lock_guard<std::mutex> lock(S().mu);
  std::vector<Region> keep;
  for (const Region &r : S().regions)
    if (r.name.rfind("static ", 0) == 0) keep.push_back(r);
  S().regions.swap(keep);
}

// launches, errors, pointer checks, extent checks since the start
void hc_counters(uint64_t *launches, uint64_t *errors, uint64_t *ptr_checks, uint64_t *extent_checks) {
  std::lock_guard<std::mutex> lock(S().mu);
  *launches = S().launches;
  *errors = S().errors;
  *ptr_checks = S().ptr_checks;
  *extent_checks = S().extent_checks;
}

// ---- registration (called by the host-only objects' static constructors) --
void **__hipRegisterFatBinary(const void *) {
  static void *handle = nullptr;
  return &handle;
}

void __hipUnregisterFatBinary(void **) {}

void __hipRegisterFunction(void **, const void *hostFunction, char *, const char *deviceName, unsigned int,
                           void *, void *, void *, void *, int *) {
  std::lock_guard<std::mutex> lock(S().mu);
  KernelInfo k;
  k.mangled = deviceName;
  S().kernels[hostFunction] = k;
}

void __hipRegisterVar(void **, void *var, char *, char *deviceVar, int, size_t size, int, int) {
  std::lock_guard<std::mutex> lock(S().mu);
  const uintptr_t p = S().next;
  S().next += (size + 65535) / 65536 * 65536 + 65536;
  const Region r{p, p + size, std::string("static ") + deviceVar};
  S().regions.push_back(r);
  S().vars[var] = r;
}

// ---- the runtime calls the library makes -------------------------------
hipError_t __hipPushCallConfiguration(dim3 grid, dim3 block, size_t shm, hipStream_t s) {
  std::lock_guard<std::mutex> lock(S().mu);
  S().cfg.push_back({grid, block, shm, s});
  return hipSuccess;
}

hipError_t __hipPopCallConfiguration(dim3 *grid, dim3 *block, size_t *shm, hipStream_t *s) {
  std::lock_guard<std::mutex> lock(S().mu);
  if (S().cfg.empty()) return hipErrorInvalidConfiguration;
  const Config c = S().cfg.back();
  S().cfg.pop_back();
  *grid = c.grid;
  *block = c.block;
  *shm = c.shm;
  *s = c.s;
  return hipSuccess;
}

hipError_t hipLaunchKernel(const void *f, dim3 grid, dim3 block, void **args, size_t shm, hipStream_t) {
  check_launch(f, grid, block, args, shm);
  return hipSuccess;
}

hipError_t hipExtLaunchKernel(const void *f, dim3 grid, dim3 block, void **args, size_t shm, hipStream_t,
                              hipEvent_t, hipEvent_t, int) {
  check_launch(f, grid, block, args, shm);
  return hipSuccess;
}

hipError_t hipGetLastError(void) {
  std::lock_guard<std::mutex> lock(S().mu);
  const hipError_t e = S().last;
  S().last = hipSuccess;
  return e;
}

const char *hipGetErrorString(hipError_t) { return "error recorded by the launch checker"; }

hipError_t hipMemcpyAsync(void *dst, const void *src, size_t bytes, hipMemcpyKind kind, hipStream_t) {
  static const KernelInfo copy{"hipMemcpyAsync", "hipMemcpyAsync", {}, {}, true, 0};
  std::lock_guard<std::mutex> lock(S().mu);
  if (kind == hipMemcpyDeviceToHost) {
    check_extent(copy, "source", src, bytes);
    std::memset(dst, 0, bytes);  // host memory: the sanitizer checks the extent
  } else if (kind == hipMemcpyDeviceToDevice) {
    check_extent(copy, "source", src, bytes);
    check_extent(copy, "destination", dst, bytes);
  } else {
    error("hipMemcpyAsync: unexpected copy kind");
  }
  return hipSuccess;
}

hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipGetDevice(int *d) {
  *d = 0;
  return hipSuccess;
}

hipError_t hipGetSymbolAddress(void **p, const void *symbol) {
  std::lock_guard<std::mutex> lock(S().mu);
  auto it = S().vars.find(symbol);
  if (it == S().vars.end()) return hipErrorInvalidSymbol;
  *p = reinterpret_cast<void *>(it->second.lo);
  return hipSuccess;
}

hipError_t hipEventCreate(hipEvent_t *e) {
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<int *>(e);
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float *ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}

// streams and events are tokens; launches run (are checked) in issue order
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned int) { return hipSuccess; }
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned int) {
  *s = reinterpret_cast<hipStream_t>(new int(3));
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t s) {
  delete reinterpret_cast<int *>(s);
  return hipSuccess;
}
hipError_t hipStreamGetDevice(hipStream_t, hipDevice_t *d) {
  *d = 0;
  return hipSuccess;
}

// recorded steps: capture records nothing here; the graph handles are tokens
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus *st) {
  *st = hipStreamCaptureStatusNone;
  return hipSuccess;
}
hipError_t hipStreamBeginCapture(hipStream_t, hipStreamCaptureMode) { return hipSuccess; }
hipError_t hipStreamEndCapture(hipStream_t, hipGraph_t *g) {
  *g = reinterpret_cast<hipGraph_t>(new int(1));
  return hipSuccess;
}
hipError_t hipGraphInstantiate(hipGraphExec_t *x, hipGraph_t, hipGraphNode_t *, char *, size_t) {
  *x = reinterpret_cast<hipGraphExec_t>(new int(2));
  return hipSuccess;
}
hipError_t hipGraphLaunch(hipGraphExec_t, hipStream_t) { return hipSuccess; }
hipError_t hipGraphDestroy(hipGraph_t g) {
  delete reinterpret_cast<int *>(g);
  return hipSuccess;
}
hipError_t hipGraphExecDestroy(hipGraphExec_t x) {
  delete reinterpret_cast<int *>(x);
  return hipSuccess;
}

}  // extern "C"

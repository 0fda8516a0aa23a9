// C-ABI entry points of the 2M + Ozaki-II library (declared in include/o2m.h).
//
// Every call validates its arguments on the host, then enqueues on the
// caller's stream:
//   K1  per-row / per-column maxima and exponents      (Algorithm 1, step 2;
//       the Cauchy-Schwarz rule adds a sum-of-squares pass)
//   K2  quantize, residues and 2M pre into int8 planes (steps 3-4, eq. 2m-pre)
//   K3  batched int8 MFMA GEMMs, C mod m as int8       (step 4, eq. 2m-mul)
//   K4  2M post, CRT, symmetric lift, descale          (steps 4-7, eq. 2m-post)
// and returns without synchronizing.
#include <algorithm>
#include <atomic>
#include <map>
#include <math.h>
#include <mutex>
#include <stdio.h>
#include <string.h>

#include "o2m.h"
#include "o2m_internal.h"

using namespace o2m;

namespace {

constexpr int kMaxDevices = 64;
constexpr int kPhaseCount = 4;
constexpr int kMaxTimedCalls = 1024;

// Scratch memory of the calls on one stream of one device.  Calls on the same
// stream run one after another, so they can share it; calls on different
// streams never do.
struct StreamState {
    void *ws = nullptr;       // library-owned workspace
    size_t ws_bytes = 0;
    void *user_ws = nullptr;  // caller-owned workspace (if set)
    size_t user_bytes = 0;
};

std::mutex g_mu;
std::map<std::pair<int, hipStream_t>, StreamState> g_streams;

// The device status word: a static device array (one per GPU), whose address
// on each device is looked up once with that device current.
__device__ __align__(256) int status_word[64];
int *g_status[kMaxDevices];

// Scratch memory of zgemm_2m_noalloc: a static device array, one per GPU
// (every GPU the library's code is loaded on holds its copy until the
// process ends, 256 MiB, whether or not the call is used).  In
// host code `scratch` only stands in for the symbol; its device address on
// each GPU is looked up once, with that GPU current, and kept in
// g_scratch[device].  Every zgemm_2m_noalloc call on a GPU uses that GPU's
// array, so such calls that overlap in time on one GPU race.
constexpr size_t kScratchBytes = (size_t)O2M_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
void *g_scratch[kMaxDevices];

// phase timing (its own lock: every call takes a slot of events)
std::mutex g_tmu;
std::atomic<bool> g_timing{false};
hipEvent_t g_events[kMaxTimedCalls][kPhaseCount + 1];
bool g_events_made[kMaxTimedCalls];
int g_timed_calls = 0;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base((char *)b) {}
    void *take(size_t bytes) {
        void *p = base ? base + off : nullptr;
        off += align256(bytes);
        return p;
    }
};

int floor_half(int P) { return P >= 0 ? P / 2 : -((-P + 1) / 2); }

// Geometry of one call
struct Geometry {
    int rows_a, rows_b;       // operand rows (m and n; HERK/SYRK/rank-2k: n and n)
    int k;                    // inner dimension of one source (SYRK: ceil(k/2))
    int a_pad, b_pad, kpad, kblocks;  // kblocks: of one source
    int halves;               // 2 for rank-2k updates ([A|B] along k), else 1
    size_t plane_a, plane_b, plane_c;
    int products;             // int8 GEMMs: 2 per 2M modulus, 3 per 3M modulus
                              // (GEMM), 1 per modulus (HERK/SYRK/rank-2k)
    int planes;               // operand planes per side: products (GEMM), 2N (symmetric)
    bool shared_planes;       // symmetric ops: B planes are the A- planes
    int kscan;                // columns of A (rows of B) that K1 walks: the call's k
    int cs_ca, cs_cb;         // Cauchy-Schwarz chunks per row of A (one source) / column of B
};

// 2M moduli among the first N (the rest are the 3M extension of a hybrid set)
int count_2m(int N) { return N < kMax2M ? N : kMax2M; }

Geometry make_geometry(int rows_a, int rows_b, int k, int N, bool sym, int halves, int kscan) {
    Geometry g;
    g.rows_a = rows_a;
    g.rows_b = rows_b;
    g.k = k;
    g.a_pad = round_up(rows_a > 0 ? rows_a : 1, kRowBlock);
    g.b_pad = round_up(rows_b > 0 ? rows_b : 1, kRowBlock);
    g.kpad = round_up(k > 0 ? k : 1, kStageK);
    g.kblocks = g.kpad / kStageK;
    g.halves = halves;
    g.plane_a = (size_t)g.a_pad * g.kpad * halves;
    g.plane_b = (size_t)g.b_pad * g.kpad;
    g.plane_c = (size_t)g.a_pad * g.b_pad;
    const int n2 = count_2m(N);
    g.products = sym ? N : 2 * n2 + 3 * (N - n2);
    g.planes = sym ? 2 * N : g.products;
    g.shared_planes = sym;
    g.kscan = kscan;
    // room for either layout of a GEMM operand (rows of a column-major matrix,
    // or columns when it is transposed); symmetric ops read rows only
    g.cs_ca = sym ? cs_chunks(0, rows_a, kscan) : std::max(cs_chunks(0, rows_a, kscan), cs_chunks(1, kscan, rows_a));
    g.cs_cb = sym ? 0 : std::max(cs_chunks(1, kscan, rows_b), cs_chunks(0, rows_b, kscan));
    return g;
}

struct Buffers {
    unsigned long long *amax_a, *amax_b;
    unsigned *queue;  // the int8 GEMM's slot counters
    int32_t *E, *F;
    CsPartials csa, csb;  // Cauchy-Schwarz chunk records (rows of A, columns of B)
    int8_t *planes_a, *planes_b, *res;
};

CsPartials cs_partials(Carver &c, int chunks, int pitch) {
    CsPartials p;
    const size_t bytes = sizeof(unsigned long long) * (size_t)chunks * pitch;
    p.mx = (unsigned long long *)c.take(bytes);
    p.s2 = (unsigned long long *)c.take(bytes);
    p.s1n = (unsigned long long *)c.take(bytes);
    p.pitch = pitch;
    p.chunks = chunks;
    return p;
}

size_t carve(const Geometry &g, int N, void *base, Buffers *b) {
    Carver c(base);
    Buffers t;
    // amax_a, amax_b and queue stay contiguous and in this order, ending
    // where E begins: K1 clears them with one fill
    t.amax_a = (unsigned long long *)c.take(sizeof(unsigned long long) * g.a_pad);
    t.amax_b = g.shared_planes ? t.amax_a : (unsigned long long *)c.take(sizeof(unsigned long long) * g.b_pad);
    t.queue = (unsigned *)c.take(sizeof(unsigned) * 8 * kQueueStride);
    t.E = (int32_t *)c.take(sizeof(int32_t) * g.a_pad);
    t.F = g.shared_planes ? t.E : (int32_t *)c.take(sizeof(int32_t) * g.b_pad);
    // every record the combine step reads is written by the scan: no fill
    t.csa = cs_partials(c, g.cs_ca * g.halves, g.a_pad);
    t.csb = cs_partials(c, g.cs_cb, g.b_pad);
    t.planes_a = (int8_t *)c.take(g.plane_a * g.planes);
    t.planes_b = g.shared_planes ? t.planes_a : (int8_t *)c.take(g.plane_b * g.planes);
    t.res = (int8_t *)c.take(g.plane_c * g.products);
    if (b) *b = t;
    return c.off;
}

o2m_status hip_fail(hipError_t e) {
    if (e == hipSuccess) return O2M_OK;
    if (getenv("O2M_LOG")) fprintf(stderr, "o2m: HIP error %d (%s)\n", (int)e, hipGetErrorString(e));
    return O2M_ERR_HIP;
}

#define O2M_TRY(expr)                                        \
    do {                                                     \
        hipError_t e_ = (expr);                              \
        if (e_ != hipSuccess) return hip_fail(e_);           \
    } while (0)

// The status word of the current device (looked up on first use, under g_mu).
o2m_status status_of(int dev, int **out) {
    if (!g_status[dev]) {
        void *p = nullptr;
        O2M_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(status_word)));
        g_status[dev] = (int *)p;
    }
    *out = g_status[dev];
    return O2M_OK;
}

o2m_status current_device(int *dev) {
    O2M_TRY(hipGetDevice(dev));
    return *dev >= 0 && *dev < kMaxDevices ? O2M_OK : O2M_ERR_HIP;
}

// The static scratch array of the current device as the workspace of a call
// that must not allocate (looked up on the device's first such call).
o2m_status static_scratch(size_t bytes, void **out, int **status) {
    if (bytes > kScratchBytes) return O2M_ERR_SCRATCH;
    int dev = 0;
    o2m_status s = current_device(&dev);
    if (s != O2M_OK) return s;
    std::lock_guard<std::mutex> lock(g_mu);
    s = status_of(dev, status);
    if (s != O2M_OK) return s;
    if (!g_scratch[dev]) {
        void *p = nullptr;
        O2M_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return O2M_OK;
}

// Returns a device buffer of at least `bytes` for calls on stream st of the
// current device: the caller's buffer bound to that stream, else the
// library's buffer of that stream (allocated, or grown once the calls already
// enqueued on st have finished).
o2m_status workspace(hipStream_t st, size_t bytes, void **out, int **status) {
    int dev = 0;
    o2m_status s = current_device(&dev);
    if (s != O2M_OK) return s;
    std::lock_guard<std::mutex> lock(g_mu);
    s = status_of(dev, status);
    if (s != O2M_OK) return s;
    StreamState &d = g_streams[std::make_pair(dev, st)];
    if (d.user_ws) {
        if (d.user_bytes < bytes) return O2M_ERR_WORKSPACE;
        *out = d.user_ws;
        return O2M_OK;
    }
    if (d.ws_bytes < bytes) {
        // a stream under graph capture can neither wait nor allocate: its
        // workspace must be sized before the capture
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        O2M_TRY(hipStreamIsCapturing(st, &cs));
        if (cs != hipStreamCaptureStatusNone) return O2M_ERR_WORKSPACE;
        // earlier calls on this stream may still use the old buffer
        O2M_TRY(hipStreamSynchronize(st));
        if (d.ws) O2M_TRY(hipFree(d.ws));
        d.ws = nullptr;
        d.ws_bytes = 0;
        if (hipMalloc(&d.ws, bytes) != hipSuccess) {
            (void)hipGetLastError();
            d.ws = nullptr;
            return O2M_ERR_NOMEM;
        }
        d.ws_bytes = bytes;
    }
    *out = d.ws;
    return O2M_OK;
}

// Reserves the events of one timed call: its slot, or -1 when timing is off
// or the table is full.
int phase_begin() {
    if (!g_timing.load()) return -1;
    std::lock_guard<std::mutex> lock(g_tmu);
    if (!g_timing.load() || g_timed_calls >= kMaxTimedCalls) return -1;
    const int slot = g_timed_calls++;
    if (!g_events_made[slot]) {
        for (int p = 0; p <= kPhaseCount; ++p) (void)hipEventCreate(&g_events[slot][p]);
        g_events_made[slot] = true;
    }
    return slot;
}

void phase_mark(int slot, int phase, hipStream_t st) {
    if (slot >= 0) (void)hipEventRecord(g_events[slot][phase], st);
}

enum Op { kOpZ, kOpC, kOpH, kOpS, kOpG, kOpR, kOpH2, kOpS2 };

struct Call {
    Op op;
    int m, n, k;
    const void *A; int lda;
    const void *B; int ldb;
    void *C; int ldc;
    int N;
    int scaling;
    hipStream_t st;
    int8_t *res_out;
    int32_t *E_out, *F_out;
    bool noalloc = false;     // workspace = the static scratch array
    char ta = 'N', tb = 'N';  // GEMM operands: op(X) = X, X^T or X^H ('N', 'T', 'C')
    bool upper = false;       // symmetric ops: write the upper triangle
};

bool is_sym(Op op) { return op == kOpH || op == kOpS || op == kOpH2 || op == kOpS2; }
bool is_rank2(Op op) { return op == kOpH2 || op == kOpS2; }
bool is_real_split(Op op) { return op == kOpS || op == kOpS2; }  // SYRK-type: Z = A1 + i A2

// Inner dimension of one source after the SYRK split, and of the int8 GEMMs.
int source_k(Op op, int k) { return is_real_split(op) ? (k + 1) / 2 : k; }
int gemm_k(Op op, int k) { return (is_rank2(op) ? 2 : 1) * source_k(op, k); }

// Quantization shifts of the chosen rule for the inner dimension kin.
o2m_status shifts(const ModuliTable *t, Op op, int kin, int scaling, int *pA, int *pB) {
    const bool sym = is_sym(op);
    if (op == kOpG) { *pA = *pB = 0; return O2M_OK; }
    if (scaling == O2M_SCALE_CS) {
        return budget_cs(t, kin, sym, pA, pB) ? O2M_OK : O2M_ERR_SCALING;
    }
    if (scaling != O2M_SCALE_MAX) return O2M_ERR_SCALING;
    const int P = budget(t, kin);
    *pA = floor_half(P);
    *pB = sym ? *pA : P - *pA;
    return O2M_OK;
}

// Every quantized value is below 2^p (max rule) or 2^p + sqrt(k/2) < 2^(p+1)
// (Cauchy-Schwarz rule): the residue kernel's digit count follows.
int digits(int scaling, int p) { return residue_digits(scaling == O2M_SCALE_CS ? p + 1 : p); }

o2m_status run(const Call &c) {
    const bool sym = is_sym(c.op);
    const bool two = is_rank2(c.op);
    const bool cs = c.scaling == O2M_SCALE_CS;
    const int kc = source_k(c.op, c.k);
    const ModuliTable *t = moduli_table(c.N);
    if (!t) return O2M_ERR_NMODULI;
    int pA = 0, pB = 0;
    o2m_status s = shifts(t, c.op, gemm_k(c.op, c.k), c.scaling, &pA, &pB);
    if (s != O2M_OK) return s;
    const Geometry g = make_geometry(c.m, sym ? c.m : c.n, kc, c.N, sym, two ? 2 : 1, c.k);
    if ((long)g.a_pad * g.b_pad > (1L << 40) || (long)g.a_pad / kRowBlock * (g.b_pad / kRowBlock) * g.products > 0x7FFFFFFFL)
        return O2M_ERR_SIZE;
    void *ws = nullptr;
    int *status = nullptr;
    const size_t need = carve(g, c.N, nullptr, nullptr);
    s = c.noalloc ? static_scratch(need, &ws, &status) : workspace(c.st, need, &ws, &status);
    if (s != O2M_OK) return s;
    Buffers b;
    carve(g, c.N, ws, &b);

    const ElemType et = c.op == kOpC ? kF32 : c.op == kOpG ? kI32 : is_real_split(c.op) ? kR64 : kF64;

    const int slot = phase_begin();
    phase_mark(slot, 0, c.st);
    // ---- K1: maxima and exponents (rank-2k: row i of A and of B share one) --
    // the maxima (max rule) and the GEMM's slot counters start at zero: one
    // fill over the contiguous amax_a .. queue region of the workspace (carve
    // order)
    O2M_TRY(launch_zero(b.amax_a, (size_t)((char *)b.E - (char *)b.amax_a), c.st));
    // where the operand rows sit: A's rows are rows of the stored A (mode 0)
    // or, transposed, its columns (mode 1); B's operand rows (the columns of
    // op(B)) are columns of the stored B (mode 1) or, transposed, its rows
    const int amode = c.ta == 'N' ? 0 : 1, bmode = c.tb == 'N' ? 1 : 0;
    const int a_rows = amode == 0 ? c.m : c.k, a_cols = amode == 0 ? c.k : c.m;  // stored A
    const int b_rows = bmode == 1 ? c.k : c.n, b_cols = bmode == 1 ? c.n : c.k;  // stored B
    if (cs && c.op != kOpG) {
        // one pass over each operand: chunk records, then the exponents they
        // settle (the few entries they leave open are summed from the data)
        b.csa.chunks = cs_chunks(amode, a_rows, a_cols) * g.halves;
        b.csb.chunks = sym ? 0 : cs_chunks(bmode, b_rows, b_cols);
        O2M_TRY(launch_cs_scan(amode, et, a_rows, a_cols, c.A, c.lda, b.csa, 0, c.st));
        if (two) O2M_TRY(launch_cs_scan(0, et, c.m, c.k, c.B, c.ldb, b.csa, b.csa.chunks / 2, c.st));
        if (!sym) O2M_TRY(launch_cs_scan(bmode, et, b_rows, b_cols, c.B, c.ldb, b.csb, 0, c.st));
        CsCombineArgs cg;
        memset(&cg, 0, sizeof cg);
        cg.ca = c.m;
        cg.cb = sym ? 0 : c.n;
        cg.pa = b.csa;
        cg.pb = b.csb;
        cg.Ea = b.E;
        cg.Eb = b.F;
        cg.status = status;
        cg.A = c.A;
        cg.lda = c.lda;
        cg.B2 = two ? c.B : nullptr;
        cg.ldb2 = c.ldb;
        cg.B = sym ? nullptr : c.B;
        cg.ldb = c.ldb;
        cg.k = c.k;
        cg.amode = amode;
        cg.bmode = bmode;
        O2M_TRY(launch_cs_combine(et, cg, c.st));
    } else {
        O2M_TRY(launch_amax(amode, et, a_rows, a_cols, c.A, c.lda, b.amax_a, c.st));
        if (two) O2M_TRY(launch_amax(0, et, c.m, c.k, c.B, c.ldb, b.amax_a, c.st));
        if (!sym) O2M_TRY(launch_amax(bmode, et, b_rows, b_cols, c.B, c.ldb, b.amax_b, c.st));
        if (c.op != kOpG)
            O2M_TRY(launch_exponents(c.m, b.amax_a, b.E, sym ? 0 : c.n, b.amax_b, b.F, status, c.st));
    }
    phase_mark(slot, 1, c.st);

    // ---- K2: residues + 2M pre ---------------------------------------------
    // Rank-2k: plane 2l = [A+ | B+], plane 2l+1 = [B- | A-] along k, so that
    // one GEMM per modulus gives C+ = A+ B-^T + B+ A-^T (Section 5, HER2K).
    const int kb = g.kblocks;
    const int pkb = g.halves * kb;
    const int rmode = is_real_split(c.op) ? 2 : amode;
    const int khalf = is_real_split(c.op) ? kc : 0;
    const int32_t *Eq = c.op == kOpG ? nullptr : b.E;
    PlaneGeom ga = {c.m, kc, c.k, g.a_pad, kb, pkb, 0, two ? kb : 0, g.plane_a, c.ta == 'C'};
    O2M_TRY(launch_residues(rmode, et, c.A, c.lda, Eq, pA, digits(c.scaling, pA), khalf, ga, t->res,
                            b.planes_a, c.st));
    if (two) {
        PlaneGeom gb2 = {c.m, kc, c.k, g.a_pad, kb, pkb, kb, 0, g.plane_a};
        O2M_TRY(launch_residues(rmode, et, c.B, c.ldb, Eq, pA, digits(c.scaling, pA), khalf, gb2, t->res,
                                b.planes_a, c.st));
    }
    if (!sym) {
        PlaneGeom gb = {c.n, c.k, c.k, g.b_pad, kb, kb, 0, 0, g.plane_b, c.tb == 'C'};
        O2M_TRY(launch_residues(bmode, et, c.B, c.ldb, c.op == kOpG ? nullptr : b.F, pB, digits(c.scaling, pB), 0,
                                gb, t->res, b.planes_b, c.st));
    }
    phase_mark(slot, 2, c.st);

    // ---- K3: int8 GEMMs ----------------------------------------------------
    GemmArgs gm;
    memset(&gm, 0, sizeof gm);
    gm.a = b.planes_a;
    gm.b = sym ? b.planes_a + g.plane_a : b.planes_b;
    gm.c = b.res;
    gm.queue = b.queue;
    gm.a_pstride = sym ? 2 * g.plane_a : g.plane_a;
    gm.b_pstride = sym ? 2 * g.plane_a : g.plane_b;
    gm.c_pstride = g.plane_c;
    gm.mt = g.a_pad / kRowBlock;
    gm.nt = g.b_pad / kRowBlock;
    gm.kblocks = pkb;
    gm.batch = g.products;
    gm.ldc = g.a_pad;
    for (int p = 0; p < g.products; ++p) {   // product -> modulus
        const int n2 = t->res.n2;
        const int l = sym ? p : p < 2 * n2 ? p >> 1 : n2 + (p - 2 * n2) / 3;
        gm.mod[p] = t->res.mod[l];
        gm.inv[p] = t->res.inv[l];
    }
    O2M_TRY(launch_gemm(gm, c.st));
    phase_mark(slot, 3, c.st);

    // ---- K4: 2M post + CRT + lift + descale ---------------------------------
    CrtArgs ca;
    memset(&ca, 0, sizeof ca);
    ca.res = b.res;
    ca.plane_bytes = g.plane_c;
    ca.ldr = g.a_pad;
    ca.m = c.m;
    ca.n = sym ? c.m : c.n;
    ca.c = c.op == kOpR ? (void *)c.res_out : c.C;
    ca.ldc = c.ldc;
    ca.E = b.E;
    ca.F = sym ? b.E : b.F;
    ca.scale_bias = -(pA + pB);
    ca.amaxA = b.amax_a;
    ca.amaxB = b.amax_b;
    ca.k = c.k;
    ca.status = status;
    ca.upper = c.upper;
    for (int l = 0; l < c.N; ++l) {
        ca.hmod[l] = (short)t->res.mod[l];
        ca.hroot[l] = (short)t->res.root[l];
    }
    int mode = 0;
    ElemType ot = kF64;
    switch (c.op) {
    case kOpZ: mode = 0; break;
    case kOpC: mode = 0; ot = kF32; break;
    case kOpH: case kOpH2: mode = 1; break;
    case kOpS: case kOpS2: mode = 2; break;
    case kOpG: mode = 3; break;
    case kOpR: mode = 4; break;
    }
    O2M_TRY(launch_crt(mode, ot, ca, t->crt, c.st));
    if (c.op == kOpR) {
        if (c.E_out) O2M_TRY(hipMemcpyAsync(c.E_out, b.E, sizeof(int32_t) * c.m, hipMemcpyDeviceToDevice, c.st));
        if (c.F_out) O2M_TRY(hipMemcpyAsync(c.F_out, b.F, sizeof(int32_t) * c.n, hipMemcpyDeviceToDevice, c.st));
    }
    phase_mark(slot, 4, c.st);
    if (getenv("O2M_LOG"))
        fprintf(stderr, "o2m: op=%d m=%d n=%d k=%d N=%d scaling=%d log2M=%.2f pA=%d pB=%d T=%d ws=%zu\n",
                (int)c.op, c.m, c.n, c.k, c.N, c.scaling, t->log2M, pA, pB, t->crt.limbs, need);
    return O2M_OK;
}

// BLAS-style argument checks shared by the GEMM-shaped calls
o2m_status check_gemm(int m, int n, int k, const void *A, int lda, const void *B, int ldb, const void *C,
                      int ldc, int N, int maxN) {
    if (m < 0) return -1;
    if (n < 0) return -2;
    if (k < 0) return -3;
    if (!A && m > 0 && k > 0) return -4;
    if (lda < (m > 1 ? m : 1)) return -5;
    if (!B && k > 0 && n > 0) return -6;
    if (ldb < (k > 1 ? k : 1)) return -7;
    if (!C && m > 0 && n > 0) return -8;
    if (ldc < (m > 1 ? m : 1)) return -9;
    if (N < 1 || N > maxN) return O2M_ERR_NMODULI;
    if (k > (N > O2M_MAX_MODULI ? O2M_MAX_K_HYBRID : O2M_MAX_K)) return O2M_ERR_KLIMIT;
    return O2M_OK;
}

o2m_status check_sym(char uplo, int n, int k, const void *A, int lda, const void *C, int ldc, int N) {
    if (uplo != 'L' && uplo != 'l' && uplo != 'U' && uplo != 'u') return -1;
    if (n < 0) return -2;
    if (k < 0) return -3;
    if (!A && n > 0 && k > 0) return -4;
    if (lda < (n > 1 ? n : 1)) return -5;
    if (!C && n > 0) return -6;
    if (ldc < (n > 1 ? n : 1)) return -7;
    if (N < 1 || N > O2M_MAX_MODULI) return O2M_ERR_NMODULI;
    if (k > O2M_MAX_K) return O2M_ERR_KLIMIT;
    return O2M_OK;
}

// rank-2k: the GEMMs run over [A | B], so twice the (SYRK-split) k must fit
o2m_status check_sym2(char uplo, int n, int k, const void *A, int lda, const void *B, int ldb, const void *C,
                      int ldc, int N, bool split) {
    if (uplo != 'L' && uplo != 'l' && uplo != 'U' && uplo != 'u') return -1;
    if (n < 0) return -2;
    if (k < 0) return -3;
    if (!A && n > 0 && k > 0) return -4;
    if (lda < (n > 1 ? n : 1)) return -5;
    if (!B && n > 0 && k > 0) return -6;
    if (ldb < (n > 1 ? n : 1)) return -7;
    if (!C && n > 0) return -8;
    if (ldc < (n > 1 ? n : 1)) return -9;
    if (N < 1 || N > O2M_MAX_MODULI) return O2M_ERR_NMODULI;
    const long kin = 2L * (split ? (k + 1) / 2 : k);
    if (kin > O2M_MAX_K) return O2M_ERR_KLIMIT;
    return O2M_OK;
}

o2m_status check_scaling(int scaling) {
    return scaling == O2M_SCALE_MAX || scaling == O2M_SCALE_CS ? O2M_OK : O2M_ERR_SCALING;
}

bool op_of(char op, Op *out) {
    switch (op) {
    case 'z': *out = kOpZ; return true;
    case 'c': *out = kOpC; return true;
    case 'h': *out = kOpH; return true;
    case 's': *out = kOpS; return true;
    case 'g': *out = kOpG; return true;
    case 'r': *out = kOpR; return true;
    case 'x': *out = kOpH2; return true;
    case 'y': *out = kOpS2; return true;
    default: return false;
    }
}

// 'N', 'T' or 'C' (either case) as upper case; 0 for anything else
char trans_of(char t) {
    switch (t) {
    case 'n': case 'N': return 'N';
    case 't': case 'T': return 'T';
    case 'c': case 'C': return 'C';
    default: return 0;
    }
}

o2m_status check_gemm_op(char ta, char tb, int m, int n, int k, const void *A, int lda, const void *B, int ldb,
                         const void *C, int ldc, int N, int maxN) {
    if (!trans_of(ta)) return -1;
    if (!trans_of(tb)) return -2;
    if (m < 0) return -3;
    if (n < 0) return -4;
    if (k < 0) return -5;
    const int arows = trans_of(ta) == 'N' ? m : k, brows = trans_of(tb) == 'N' ? k : n;
    if (!A && m > 0 && k > 0) return -6;
    if (lda < (arows > 1 ? arows : 1)) return -7;
    if (!B && k > 0 && n > 0) return -8;
    if (ldb < (brows > 1 ? brows : 1)) return -9;
    if (!C && m > 0 && n > 0) return -10;
    if (ldc < (m > 1 ? m : 1)) return -11;
    if (N < 1 || N > maxN) return O2M_ERR_NMODULI;
    if (k > (N > O2M_MAX_MODULI ? O2M_MAX_K_HYBRID : O2M_MAX_K)) return O2M_ERR_KLIMIT;
    return O2M_OK;
}

o2m_status gemm_op(Op op, char transa, char transb, int m, int n, int k, const void *A, int lda, const void *B,
                   int ldb, void *C, int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_gemm_op(transa, transb, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_MAX_MODULI_HYBRID);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    Call c{op, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr, nullptr, nullptr};
    c.ta = trans_of(transa);
    c.tb = trans_of(transb);
    return run(c);
}

}  // namespace

extern "C" {

o2m_status zgemm_2m_ex(int m, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                       int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_gemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_MAX_MODULI_HYBRID);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    return run(Call{kOpZ, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr});
}

o2m_status zgemm_2m_noalloc(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                            double *C, int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_gemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_MAX_MODULI_HYBRID);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    Call c{kOpZ, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr, nullptr, nullptr};
    c.noalloc = true;
    return run(c);
}

o2m_status zgemm_2m(int m, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                    int ldc, int n_moduli, void *stream) {
    return zgemm_2m_ex(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status zgemm_2m_op(char transa, char transb, int m, int n, int k, const double *A, int lda, const double *B,
                       int ldb, double *C, int ldc, int n_moduli, int scaling, void *stream) {
    return gemm_op(kOpZ, transa, transb, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, stream);
}

o2m_status cgemm_2m_op(char transa, char transb, int m, int n, int k, const float *A, int lda, const float *B,
                       int ldb, float *C, int ldc, int n_moduli, int scaling, void *stream) {
    return gemm_op(kOpC, transa, transb, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, stream);
}

o2m_status cgemm_2m_ex(int m, int n, int k, const float *A, int lda, const float *B, int ldb, float *C,
                       int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_gemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_MAX_MODULI_HYBRID);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    return run(Call{kOpC, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr});
}

o2m_status cgemm_2m(int m, int n, int k, const float *A, int lda, const float *B, int ldb, float *C,
                    int ldc, int n_moduli, void *stream) {
    return cgemm_2m_ex(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status zherk_2m_ex(char uplo, int n, int k, const double *A, int lda, double *C, int ldc, int n_moduli,
                       int scaling, void *stream) {
    o2m_status s = check_sym(uplo, n, k, A, lda, C, ldc, n_moduli);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || n == 0) return s;
    Call c{kOpH, n, n, k, A, lda, nullptr, 1, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr};
    c.upper = uplo == 'U' || uplo == 'u';
    return run(c);
}

o2m_status zherk_2m(char uplo, int n, int k, const double *A, int lda, double *C, int ldc, int n_moduli,
                    void *stream) {
    return zherk_2m_ex(uplo, n, k, A, lda, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status dsyrk_2m_ex(char uplo, int n, int k, const double *A, int lda, double *C, int ldc, int n_moduli,
                       int scaling, void *stream) {
    o2m_status s = check_sym(uplo, n, k, A, lda, C, ldc, n_moduli);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || n == 0) return s;
    Call c{kOpS, n, n, k, A, lda, nullptr, 1, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr};
    c.upper = uplo == 'U' || uplo == 'u';
    return run(c);
}

o2m_status dsyrk_2m(char uplo, int n, int k, const double *A, int lda, double *C, int ldc, int n_moduli,
                    void *stream) {
    return dsyrk_2m_ex(uplo, n, k, A, lda, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status zher2k_2m_ex(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                        int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_sym2(uplo, n, k, A, lda, B, ldb, C, ldc, n_moduli, false);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || n == 0) return s;
    Call c{kOpH2, n, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr};
    c.upper = uplo == 'U' || uplo == 'u';
    return run(c);
}

o2m_status zher2k_2m(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                     int ldc, int n_moduli, void *stream) {
    return zher2k_2m_ex(uplo, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status dsyr2k_2m_ex(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                        int ldc, int n_moduli, int scaling, void *stream) {
    o2m_status s = check_sym2(uplo, n, k, A, lda, B, ldb, C, ldc, n_moduli, true);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || n == 0) return s;
    Call c{kOpS2, n, n, k, A, lda, B, ldb, C, ldc, n_moduli, scaling, (hipStream_t)stream, nullptr,
                    nullptr, nullptr};
    c.upper = uplo == 'U' || uplo == 'u';
    return run(c);
}

o2m_status dsyr2k_2m(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb, double *C,
                     int ldc, int n_moduli, void *stream) {
    return dsyr2k_2m_ex(uplo, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_SCALE_MAX, stream);
}

o2m_status gauss_gemm_2m(int m, int n, int k, const int32_t *A, int lda, const int32_t *B, int ldb,
                         int64_t *C, int ldc, int n_moduli, void *stream) {
    o2m_status s = check_gemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli, 8);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    return run(Call{kOpG, m, n, k, A, lda, B, ldb, C, ldc, n_moduli, O2M_SCALE_MAX, (hipStream_t)stream, nullptr,
                    nullptr, nullptr});
}

o2m_status zgemm_2m_residues_ex(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                                int n_moduli, int scaling, int8_t *res, int32_t *E, int32_t *F, void *stream) {
    o2m_status s = check_gemm(m, n, k, A, lda, B, ldb, res, m > 1 ? m : 1, n_moduli, O2M_MAX_MODULI_HYBRID);
    if (s == O2M_OK) s = check_scaling(scaling);
    if (s != O2M_OK || m == 0 || n == 0) return s;
    return run(Call{kOpR, m, n, k, A, lda, B, ldb, nullptr, m, n_moduli, scaling, (hipStream_t)stream, res, E, F});
}

o2m_status zgemm_2m_residues(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                             int n_moduli, int8_t *res, int32_t *E, int32_t *F, void *stream) {
    return zgemm_2m_residues_ex(m, n, k, A, lda, B, ldb, n_moduli, O2M_SCALE_MAX, res, E, F, stream);
}

o2m_status o2m_moduli(int n_moduli, int32_t *m_out, int32_t *s_out, double *log2M_out) {
    if (n_moduli < 1 || n_moduli > O2M_MAX_MODULI_HYBRID) return O2M_ERR_NMODULI;
    const ModuliTable *t = moduli_table(n_moduli);
    for (int l = 0; l < n_moduli; ++l) {
        if (m_out) m_out[l] = t->res.mod[l];
        if (s_out) s_out[l] = t->res.root[l];
    }
    if (log2M_out) *log2M_out = t->log2M;
    return O2M_OK;
}

o2m_status o2m_budget(int n_moduli, int k, int *P_out) {
    if (n_moduli < 1 || n_moduli > O2M_MAX_MODULI_HYBRID) return O2M_ERR_NMODULI;
    if (k < 0) return -2;
    if (!P_out) return -3;
    *P_out = budget(moduli_table(n_moduli), k);
    return O2M_OK;
}


o2m_status o2m_shifts(char op, int n_moduli, int k, int scaling, int *pA_out, int *pB_out) {
    Op o;
    if (!op_of(op, &o)) return -1;
    if (n_moduli < 1 || n_moduli > (is_sym(o) ? O2M_MAX_MODULI : O2M_MAX_MODULI_HYBRID)) return O2M_ERR_NMODULI;
    if (k < 0) return -3;
    if (!pA_out || !pB_out) return -5;
    if (check_scaling(scaling) != O2M_OK) return O2M_ERR_SCALING;
    return shifts(moduli_table(n_moduli), o, gemm_k(o, k), scaling, pA_out, pB_out);
}

size_t o2m_workspace_bytes(char op, int m, int n, int k, int n_moduli) {
    Op o;
    if (!op_of(op, &o) || n_moduli < 1 || m < 0 || n < 0 || k < 0) return 0;
    if (n_moduli > (is_sym(o) ? O2M_MAX_MODULI : o == kOpG ? 8 : O2M_MAX_MODULI_HYBRID)) return 0;
    const bool sym = is_sym(o);
    const Geometry g = make_geometry(m, sym ? m : n, source_k(o, k), n_moduli, sym, is_rank2(o) ? 2 : 1, k);
    return carve(g, n_moduli, nullptr, nullptr);
}

o2m_status o2m_set_workspace(void *dev_ptr, size_t bytes, void *stream) {
    int dev = 0;
    if (current_device(&dev) != O2M_OK) return O2M_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    StreamState &d = g_streams[std::make_pair(dev, (hipStream_t)stream)];
    d.user_ws = dev_ptr;
    d.user_bytes = dev_ptr ? bytes : 0;
    return O2M_OK;
}

o2m_status o2m_release_workspace(void *stream) {
    int dev = 0;
    if (current_device(&dev) != O2M_OK) return O2M_ERR_HIP;
    hipStream_t st = (hipStream_t)stream;
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_streams.find(std::make_pair(dev, st));
    if (it == g_streams.end() || !it->second.ws) return O2M_OK;
    if (hipStreamSynchronize(st) != hipSuccess) return O2M_ERR_HIP;
    if (hipFree(it->second.ws) != hipSuccess) return O2M_ERR_HIP;
    it->second.ws = nullptr;
    it->second.ws_bytes = 0;
    return O2M_OK;
}

o2m_status o2m_get_status(void *stream, int *device_status) {
    if (!device_status) return -2;
    int dev = 0;
    if (current_device(&dev) != O2M_OK) return O2M_ERR_HIP;
    hipStream_t st = (hipStream_t)stream;
    if (hipStreamSynchronize(st) != hipSuccess) return O2M_ERR_HIP;
    int *p = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        if (status_of(dev, &p) != O2M_OK) return O2M_ERR_HIP;
    }
    if (hipMemcpy(device_status, p, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess) return O2M_ERR_HIP;
    if (launch_zero(p, sizeof(int), st) != hipSuccess) return O2M_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return O2M_ERR_HIP;
    return O2M_OK;
}

o2m_status o2m_phase_timing(int enable) {
    std::lock_guard<std::mutex> lock(g_tmu);
    g_timing.store(enable != 0);
    g_timed_calls = 0;
    return O2M_OK;
}

int o2m_phase_times(float *ms, int max_phases) {
    if (!ms || max_phases < 0) return -1;
    std::lock_guard<std::mutex> lock(g_tmu);
    const int n = g_timed_calls;
    int count = kPhaseCount < max_phases ? kPhaseCount : max_phases;
    for (int p = 0; p < count; ++p) ms[p] = 0.0f;
    if (n == 0) return 0;
    if (hipEventSynchronize(g_events[n - 1][kPhaseCount]) != hipSuccess) return -1;
    for (int c = 0; c < n; ++c)
        for (int p = 0; p < count; ++p) {
            float t = 0.0f;
            if (hipEventElapsedTime(&t, g_events[c][p], g_events[c][p + 1]) != hipSuccess) return -1;
            ms[p] += t / (float)n;
        }
    return count;
}

const char *o2m_status_string(o2m_status s) {
    switch (s) {
    case O2M_OK: return "success";
    case O2M_ERR_NMODULI: return "n_moduli out of range (1..32 for GEMM, 1..22 for HERK/SYRK/rank-2k, 1..8 gauss)";
    case O2M_ERR_KLIMIT: return "k exceeds 149130 (131071 with more than 22 moduli): int32 accumulation bound";
    case O2M_ERR_WORKSPACE: return "workspace too small (a caller buffer, or a stream under graph capture whose workspace was not sized before the capture)";
    case O2M_ERR_HIP: return "HIP runtime error";
    case O2M_ERR_NOMEM: return "workspace allocation failed";
    case O2M_ERR_SIZE: return "problem too large for the tile grid";
    case O2M_ERR_SCALING: return "unknown scaling rule, or no Cauchy-Schwarz shifts for this n_moduli and k";
    case O2M_ERR_SCRATCH: return "zgemm_2m_noalloc: the call needs more than the static scratch array (O2M_NOALLOC_SCRATCH_BYTES)";
    default: break;
    }
    if (s < 0 && s >= -12) return "invalid argument (BLAS position = -status)";
    return "unknown status";
}

}  // extern "C"

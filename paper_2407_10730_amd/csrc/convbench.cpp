// convbench.cpp -- ConvBench-style benchmark harness over a CSV of convolutions.
//
// The paper's harness (Sec. III-C) is a C++ base class templated on the data type: a
// user derives from it, overrides the main convolution and (optionally) the baseline, and
// calls the execution procedure, which walks a filtered list of convolution operations
// from a CSV file, creates each one's data (random or constant values), runs warm-ups and
// measured runs of the chosen implementation (main, baseline, or a correctness check of
// main against baseline) and writes a CSV of the measured times and API call counts.
//
// Here the base class owns the walk, the device buffers and the timing; the library's
// conv2d_fwd with AUTO (the implicit / direct family) is the main convolution and the
// explicit im2col + GEMM algorithm is the baseline, as in the paper.  Times come from the
// library's per-phase breakdown (its timing tool).
//
// Input CSV: a header line naming the columns, then one convolution per line.  Columns
// (any order; the last five may be omitted):
//   name,n,c,h,w,k,r,s,stride_h,stride_w,pad_h,pad_w,dil_h,dil_w,groups[,bias][,dtype][,layout]
// dtype f32 | bf16 (y in the same type), layout nchw | nhwc, bias 0 | 1 (default 1).
//
// Usage: convbench --csv OPS.csv --out RESULTS.csv [--datagen random|constant]
//                  [--exec main|baseline|correctness] [--warmups W] [--runs R]
//                  [--seed S] [--dry-run] [--dump DIR]
// --dry-run plans every operation (no GPU needed) and writes the planner's choices.
// --dump DIR writes, per operation i, the inputs the GPU reads as raw little-endian fp32
// (DIR/i.x, i.w, i.b; x in the operation's layout, bf16 operations' values after rounding)
// and, in correctness mode, both results (i.y_main, i.y_base, fp32, in the layout), so that
// an independent checker can compare them with its own reference.
//
// Data: operation i uses seed S + i.  "random" draws x, w and bias from the SplitMix64
// streams (seed, tensor 0 / 1 / 2): stream start mix64((seed << 8) | tensor), element j =
// mix64(start + (j + 1) * 0x9E3779B97F4A7C15), value 2 * ((z >> 40) * 2^-24) - 1, exact in
// fp32 (Steele, Lea and Flood, OOPSLA 2014; Vigna's splitmix64 finaliser); "constant" sets
// x = 0.5, w = 0.25, bias = 1.
//
// Correctness mode runs main and baseline on the same data and reports the largest per-output
// difference normalised by A_o = |b_k| + sum |x * w| over the window, which the library
// itself computes as the baseline convolution of |x|, |w| and |b|.  Both results carry their
// own rounding, so the gate is twice the reference gate: 2e-5 for fp32 inputs, 2e-2 for bf16.
// A non-finite output, or a difference where A_o = 0, fails the operation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <map>
#include <sstream>
#include <string>
#include <vector>

#include "conv2d.h"

namespace {

struct Op {
    std::string name;
    conv2d_params p{};
};

const char* kPhaseNames[CONV2D_PH_COUNT] = {"pre_analysis", "pre_reorder", "in_tiling", "in_packing",
                                            "in_microkernel", "in_unpacking", "post_reorder"};

std::vector<std::string> split(const std::string& line) {
    std::vector<std::string> out;
    std::string cur;
    std::stringstream ss(line);
    while (std::getline(ss, cur, ',')) {
        size_t a = cur.find_first_not_of(" \t\r"), b = cur.find_last_not_of(" \t\r");
        out.push_back(a == std::string::npos ? std::string() : cur.substr(a, b - a + 1));
    }
    return out;
}

// Parse the convolution list; returns false (with a message) on a malformed file.
bool read_ops(const std::string& path, std::vector<Op>* ops, std::string* err) {
    std::ifstream f(path);
    if (!f) {
        *err = "cannot open " + path;
        return false;
    }
    std::string line;
    if (!std::getline(f, line)) {
        *err = "empty file";
        return false;
    }
    const std::vector<std::string> head = split(line);
    std::map<std::string, size_t> col;
    for (size_t i = 0; i < head.size(); ++i) col[head[i]] = i;
    const char* required[] = {"name", "n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w",
                              "pad_h", "pad_w", "dil_h", "dil_w", "groups"};
    for (const char* r : required)
        if (!col.count(r)) {
            *err = std::string("missing column ") + r;
            return false;
        }
    int lineno = 1;
    while (std::getline(f, line)) {
        ++lineno;
        if (line.find_first_not_of(" \t\r") == std::string::npos) continue;
        const std::vector<std::string> v = split(line);
        auto get = [&](const char* key, const char* dflt) -> std::string {
            auto it = col.find(key);
            if (it == col.end() || it->second >= v.size() || v[it->second].empty()) return dflt;
            return v[it->second];
        };
        Op op;
        op.name = get("name", "");
        conv2d_params& p = op.p;
        char* end = nullptr;
        auto num = [&](const char* key, const char* dflt, bool* ok) -> long long {
            const std::string s = get(key, dflt);
            const long long x = std::strtoll(s.c_str(), &end, 10);
            if (s.empty() || *end != '\0') *ok = false;
            return x;
        };
        bool ok = true;
        p.n = num("n", "", &ok); p.c = num("c", "", &ok); p.h = num("h", "", &ok); p.w = num("w", "", &ok);
        p.k = num("k", "", &ok); p.r = num("r", "", &ok); p.s = num("s", "", &ok);
        p.stride_h = (int32_t)num("stride_h", "", &ok); p.stride_w = (int32_t)num("stride_w", "", &ok);
        p.pad_h = (int32_t)num("pad_h", "", &ok); p.pad_w = (int32_t)num("pad_w", "", &ok);
        p.dil_h = (int32_t)num("dil_h", "", &ok); p.dil_w = (int32_t)num("dil_w", "", &ok);
        p.groups = (int32_t)num("groups", "", &ok);
        p.has_bias = (int32_t)num("bias", "1", &ok);
        const std::string dt = get("dtype", "f32"), lay = get("layout", "nchw");
        if (dt == "f32") p.x_dtype = p.y_dtype = CONV2D_F32;
        else if (dt == "bf16") p.x_dtype = p.y_dtype = CONV2D_BF16;
        else ok = false;
        if (lay == "nchw") p.layout = CONV2D_NCHW;
        else if (lay == "nhwc") p.layout = CONV2D_NHWC;
        else ok = false;
        if (!ok) {
            *err = "malformed line " + std::to_string(lineno);
            return false;
        }
        ops->push_back(op);
    }
    return true;
}

// fp32 -> bf16 bits, round to nearest even
uint16_t to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
float from_bf16(uint16_t h) {
    const uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// SplitMix64's output finaliser (Vigna, splitmix64.c).
uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Element j of the (seed, tensor) stream mapped to [-1, 1) on a 2^-23 grid.
struct Stream {
    uint64_t start;
    Stream(uint64_t seed, uint64_t tensor) : start(mix64((seed << 8) | tensor)) {}
    float at(uint64_t j) const {
        const uint64_t z = mix64(start + (j + 1) * 0x9E3779B97F4A7C15ull);
        const double u = (double)(z >> 40) * (1.0 / 16777216.0);
        return (float)(2.0 * u - 1.0);
    }
};

bool write_raw(const std::string& path, const void* data, size_t bytes) {
    FILE* f = std::fopen(path.c_str(), "wb");
    if (!f) return false;
    const bool ok = std::fwrite(data, 1, bytes, f) == bytes;
    return std::fclose(f) == 0 && ok;
}

struct Result {
    int status = CONV2D_OK;
    std::string algo;
    double op_ms = 0.0;  // mean Operation Time per call
    double phase_ms[CONV2D_PH_COUNT] = {};
    double phase_calls[CONV2D_PH_COUNT] = {};
    double tflops = 0.0;
    double max_abs_diff = -1.0, rel_diff = -1.0, err_per_point = -1.0;
    int correct = -1;
    int64_t ho = 0, wo = 0;
    conv2d_plan_info plan{};
};

// The harness.  Derive and override convolution() / convolution_baseline() to bench
// another implementation; convset_exec() walks the list.
class ConvBench {
   public:
    virtual ~ConvBench() = default;
    virtual int convolution(conv2d_desc* d, const void* x, const void* w, const float* b, void* y,
                            hipStream_t s) = 0;
    virtual int convolution_baseline(conv2d_desc* d, const void* x, const void* w, const float* b, void* y,
                                     hipStream_t s) {
        return conv2d_fwd(d, x, w, b, y, CONV2D_ALGO_IM2COL_GEMM, s);
    }
    virtual int main_algo() const = 0;

    int convset_exec(const std::vector<Op>& ops, const std::string& datagen, const std::string& exec, int warmups,
                     int runs, uint64_t seed, bool dry, const std::string& out_path, const std::string& dump);

   private:
    Result run_one(const Op& op, size_t idx, const std::string& datagen, const std::string& exec, int warmups,
                   int runs, uint64_t seed, bool dry, const std::string& dump);
};

class Conv2dBench : public ConvBench {
   public:
    int convolution(conv2d_desc* d, const void* x, const void* w, const float* b, void* y, hipStream_t s) override {
        return conv2d_fwd(d, x, w, b, y, CONV2D_ALGO_AUTO, s);
    }
    int main_algo() const override { return CONV2D_ALGO_AUTO; }
};

const char* algo_name(int a) {
    switch (a) {
        case CONV2D_ALGO_IMPLICIT_GEMM: return "implicit_gemm";
        case CONV2D_ALGO_IM2COL_GEMM: return "im2col_gemm";
        case CONV2D_ALGO_DIRECT: return "direct";
        default: return "auto";
    }
}

// Device output (fp32 or bf16) as fp32 values; false when the copy fails.
bool fetch_f32(const void* dev, int64_t n, size_t es, std::vector<float>* out) {
    out->resize(n);
    if (es == 4) return hipMemcpy(out->data(), dev, n * 4, hipMemcpyDeviceToHost) == hipSuccess;
    std::vector<uint16_t> h(n);
    if (hipMemcpy(h.data(), dev, n * 2, hipMemcpyDeviceToHost) != hipSuccess) return false;
    for (int64_t i = 0; i < n; ++i) (*out)[i] = from_bf16(h[i]);
    return true;
}

Result ConvBench::run_one(const Op& op, size_t idx, const std::string& datagen, const std::string& exec,
                          int warmups, int runs, uint64_t seed, bool dry, const std::string& dump) {
    Result r;
    conv2d_desc* d = nullptr;
    r.status = conv2d_desc_create(&op.p, &d);
    if (r.status != CONV2D_OK) return r;
    int64_t nkhw[4];
    conv2d_output_shape(d, nkhw);
    r.ho = nkhw[2];
    r.wo = nkhw[3];
    const bool baseline = exec == "baseline";
    const int algo = baseline ? CONV2D_ALGO_IM2COL_GEMM : main_algo();
    r.status = conv2d_plan_query(d, algo, &r.plan);
    r.algo = algo_name(r.plan.algo);
    const conv2d_params& p = op.p;
    const int64_t xe = p.n * p.c * p.h * p.w, we = p.k * (p.c / p.groups) * p.r * p.s;
    const int64_t ye = nkhw[0] * nkhw[1] * nkhw[2] * nkhw[3];
    const size_t es = p.x_dtype == CONV2D_BF16 ? 2 : 4, ys = p.y_dtype == CONV2D_BF16 ? 2 : 4;
    // host data, in the operation's layout: x, w, bias (random: the op's SplitMix64 streams;
    // constant: fixed values).  The random streams run over x in NCHW order, so an NHWC x holds
    // the same tensor.  bf16 operations read the values rounded to nearest even.
    std::vector<float> hx(xe), hw(we), hb(p.k);
    const uint64_t s0 = seed + idx;
    const Stream sx(s0, 0), sw(s0, 1), sb(s0, 2);
    const bool cst = datagen == "constant";
    const int64_t hw_ = p.h * p.w;
    for (int64_t i = 0; i < xe; ++i) {
        // element i in NCHW order lands at its position in the layout
        int64_t at = i;
        if (p.layout == CONV2D_NHWC) {
            const int64_t n = i / (p.c * hw_), rem = i - n * p.c * hw_, c = rem / hw_, q = rem - c * hw_;
            at = (n * hw_ + q) * p.c + c;
        }
        hx[at] = cst ? 0.5f : sx.at((uint64_t)i);
    }
    for (int64_t i = 0; i < we; ++i) hw[i] = cst ? 0.25f : sw.at((uint64_t)i);
    for (int64_t i = 0; i < p.k; ++i) hb[i] = !p.has_bias ? 0.0f : cst ? 1.0f : sb.at((uint64_t)i);
    std::vector<uint16_t> hx16, hw16;
    const void* xsrc = hx.data();
    const void* wsrc = hw.data();
    if (es == 2) {
        hx16.resize(xe);
        hw16.resize(we);
        for (int64_t i = 0; i < xe; ++i) hx[i] = from_bf16(hx16[i] = to_bf16(hx[i]));
        for (int64_t i = 0; i < we; ++i) hw[i] = from_bf16(hw16[i] = to_bf16(hw[i]));
        xsrc = hx16.data();
        wsrc = hw16.data();
    }
    const std::string stem = dump.empty() ? std::string() : dump + "/" + std::to_string(idx);
    if (!dump.empty() && (!write_raw(stem + ".x", hx.data(), xe * 4) || !write_raw(stem + ".w", hw.data(), we * 4) ||
                          !write_raw(stem + ".b", hb.data(), p.k * 4))) {
        std::fprintf(stderr, "convbench: cannot write %s.*\n", stem.c_str());
        r.status = CONV2D_E_INVALID;
    }
    if (dry || r.status != CONV2D_OK) {
        conv2d_desc_destroy(d);
        return r;
    }
    void *x = nullptr, *w = nullptr, *b = nullptr, *y = nullptr, *y2 = nullptr;
    hipStream_t s = nullptr;
    auto cleanup = [&]() {
        if (x) (void)hipFree(x);
        if (w) (void)hipFree(w);
        if (b) (void)hipFree(b);
        if (y) (void)hipFree(y);
        if (y2) (void)hipFree(y2);
        if (s) (void)hipStreamDestroy(s);
        conv2d_desc_destroy(d);
    };
    if (hipStreamCreate(&s) != hipSuccess || hipMalloc(&x, xe * es) != hipSuccess ||
        hipMalloc(&w, we * es) != hipSuccess || hipMalloc(&b, p.k * 4) != hipSuccess ||
        hipMalloc(&y, ye * ys) != hipSuccess ||
        (exec == "correctness" && hipMalloc(&y2, ye * ys) != hipSuccess) ||
        hipMemcpy(x, xsrc, xe * es, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(w, wsrc, we * es, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(b, hb.data(), p.k * 4, hipMemcpyHostToDevice) != hipSuccess) {
        r.status = CONV2D_E_ALLOC;
        cleanup();
        return r;
    }
    const float* bias = p.has_bias ? static_cast<const float*>(b) : nullptr;
    auto call = [&](bool base, void* out) {
        return base ? convolution_baseline(d, x, w, bias, out, s) : convolution(d, x, w, bias, out, s);
    };
    if (exec == "correctness") {
        // main against baseline on the same data, then A = the baseline convolution of |x|,
        // |w| and |b| (overwriting the device inputs) as the per-output denominator
        std::vector<float> ya, yb, aa;
        if ((r.status = call(false, y)) == CONV2D_OK) r.status = call(true, y2);
        if (r.status == CONV2D_OK && hipStreamSynchronize(s) != hipSuccess) r.status = CONV2D_E_HIP;
        if (r.status == CONV2D_OK && (!fetch_f32(y, ye, ys, &ya) || !fetch_f32(y2, ye, ys, &yb))) r.status = CONV2D_E_HIP;
        if (r.status == CONV2D_OK) {
            std::vector<float> ax(xe), aw(we), ab(p.k);
            for (int64_t i = 0; i < xe; ++i) ax[i] = std::fabs(hx[i]);
            for (int64_t i = 0; i < we; ++i) aw[i] = std::fabs(hw[i]);
            for (int64_t i = 0; i < p.k; ++i) ab[i] = std::fabs(hb[i]);
            std::vector<uint16_t> ax16, aw16;
            const void* axs = ax.data();
            const void* aws = aw.data();
            if (es == 2) {
                ax16.resize(xe);
                aw16.resize(we);
                for (int64_t i = 0; i < xe; ++i) ax16[i] = to_bf16(ax[i]);  // exact: |bf16| is a bf16
                for (int64_t i = 0; i < we; ++i) aw16[i] = to_bf16(aw[i]);
                axs = ax16.data();
                aws = aw16.data();
            }
            if (hipMemcpy(x, axs, xe * es, hipMemcpyHostToDevice) != hipSuccess ||
                hipMemcpy(w, aws, we * es, hipMemcpyHostToDevice) != hipSuccess ||
                hipMemcpy(b, ab.data(), p.k * 4, hipMemcpyHostToDevice) != hipSuccess)
                r.status = CONV2D_E_HIP;
            if (r.status == CONV2D_OK) r.status = call(true, y2);
            if (r.status == CONV2D_OK && (hipStreamSynchronize(s) != hipSuccess || !fetch_f32(y2, ye, ys, &aa)))
                r.status = CONV2D_E_HIP;
        }
        if (r.status == CONV2D_OK) {
            double md = 0.0, mref = 0.0, pt = 0.0;
            bool finite = true;
            for (int64_t i = 0; i < ye; ++i) {
                const double va = ya[i], vb = yb[i], a = aa[i];
                if (!std::isfinite(va) || !std::isfinite(vb) || !std::isfinite(a)) {
                    finite = false;
                    break;
                }
                const double e = std::fabs(va - vb);
                md = std::max(md, e);
                mref = std::max(mref, std::fabs(vb));
                if (a > 0) pt = std::max(pt, e / a);
                else if (e != 0) pt = HUGE_VAL;
            }
            r.max_abs_diff = finite ? md : NAN;
            r.rel_diff = finite ? (mref > 0 ? md / mref : md) : NAN;
            r.err_per_point = finite ? pt : NAN;
            const double gate = p.x_dtype == CONV2D_BF16 ? 2e-2 : 2e-5;
            r.correct = finite && pt <= gate ? 1 : 0;
            if (!dump.empty() && (!write_raw(stem + ".y_main", ya.data(), ye * 4) ||
                                  !write_raw(stem + ".y_base", yb.data(), ye * 4))) {
                std::fprintf(stderr, "convbench: cannot write %s.y_*\n", stem.c_str());
                r.correct = 0;
            }
        }
        cleanup();
        return r;
    }
    conv2d_set_timing(d, CONV2D_TIMING_OFF);
    for (int i = 0; i < warmups && r.status == CONV2D_OK; ++i) r.status = call(baseline, y);
    if (r.status == CONV2D_OK) {
        // Operation Time: an event pair around each whole call
        conv2d_set_timing(d, CONV2D_TIMING_TOTAL);
        conv2d_breakdown_reset(d);
        for (int i = 0; i < runs && r.status == CONV2D_OK; ++i) r.status = call(baseline, y);
        conv2d_breakdown_t bd{};
        if (r.status == CONV2D_OK) r.status = conv2d_breakdown(d, algo == CONV2D_ALGO_AUTO ? r.plan.algo : algo, &bd);
        if (r.status == CONV2D_OK) r.op_ms = bd.total_ms / (double)std::max<int64_t>(bd.total_calls, 1);
        // the timing tool's breakdown: an event pair around every phase launch
        conv2d_set_timing(d, CONV2D_TIMING_PHASES);
        conv2d_breakdown_reset(d);
        for (int i = 0; i < runs && r.status == CONV2D_OK; ++i) r.status = call(baseline, y);
        if (r.status == CONV2D_OK) r.status = conv2d_breakdown(d, algo == CONV2D_ALGO_AUTO ? r.plan.algo : algo, &bd);
        if (r.status == CONV2D_OK) {
            for (int ph = 0; ph < CONV2D_PH_COUNT; ++ph) {
                const double n = ph == CONV2D_PH_PRE_ANALYSIS ? 1.0 : (double)bd.fwd_calls;
                r.phase_ms[ph] = bd.ms[ph] / n;
                r.phase_calls[ph] = (double)bd.calls[ph] / n;
            }
        }
        const double flops = 2.0 * (double)ye * (double)(p.c / p.groups) * (double)(p.r * p.s);
        if (r.op_ms > 0) r.tflops = flops / (r.op_ms * 1e-3) / 1e12;
    }
    cleanup();
    return r;
}

int ConvBench::convset_exec(const std::vector<Op>& ops, const std::string& datagen, const std::string& exec,
                            int warmups, int runs, uint64_t seed, bool dry, const std::string& out_path,
                            const std::string& dump) {
    std::ofstream out(out_path);
    if (!out) {
        std::fprintf(stderr, "convbench: cannot write %s\n", out_path.c_str());
        return 2;
    }
    out << "name,n,c,h,w,k,r,s,stride_h,stride_w,pad_h,pad_w,dil_h,dil_w,groups,bias,dtype,layout,ho,wo,exec,"
           "datagen,algo,kernel,tile_m,tile_n,status,warmups,runs,op_ms,tflops";
    for (const char* ph : kPhaseNames) out << "," << ph << "_ms";
    for (const char* ph : kPhaseNames) out << "," << ph << "_calls";
    out << ",max_abs_diff,rel_diff,err_per_point,correct\n";
    int failures = 0;
    for (size_t i = 0; i < ops.size(); ++i) {
        const Op& op = ops[i];
        const Result r = run_one(op, i, datagen, exec, warmups, runs, seed, dry, dump);
        const conv2d_params& p = op.p;
        if (r.status != CONV2D_OK || r.correct == 0) ++failures;
        char buf[1024];
        std::snprintf(buf, sizeof buf,
                      "%s,%lld,%lld,%lld,%lld,%lld,%lld,%lld,%d,%d,%d,%d,%d,%d,%d,%d,%s,%s,%lld,%lld,%s,%s,%s,%d,%d,%d,"
                      "%s,%d,%d,%.6f,%.4f",
                      op.name.c_str(), (long long)p.n, (long long)p.c, (long long)p.h, (long long)p.w,
                      (long long)p.k, (long long)p.r, (long long)p.s, p.stride_h, p.stride_w, p.pad_h, p.pad_w,
                      p.dil_h, p.dil_w, p.groups, p.has_bias, p.x_dtype == CONV2D_BF16 ? "bf16" : "f32",
                      p.layout == CONV2D_NHWC ? "nhwc" : "nchw", (long long)r.ho, (long long)r.wo, exec.c_str(),
                      datagen.c_str(), r.algo.c_str(), r.plan.kernel, r.plan.tile_m, r.plan.tile_n,
                      conv2d_status_string(r.status), dry ? 0 : warmups, dry ? 0 : runs, r.op_ms, r.tflops);
        out << buf;
        for (int ph = 0; ph < CONV2D_PH_COUNT; ++ph) out << "," << r.phase_ms[ph];
        for (int ph = 0; ph < CONV2D_PH_COUNT; ++ph) out << "," << r.phase_calls[ph];
        out << "," << r.max_abs_diff << "," << r.rel_diff << "," << r.err_per_point << "," << r.correct << "\n";
        out.flush();
        std::fprintf(stderr, "[convbench] %zu/%zu %s %s %s %.4f ms%s\n", i + 1, ops.size(), op.name.c_str(),
                     exec.c_str(), conv2d_status_string(r.status), r.op_ms,
                     r.correct == 0 ? " MISMATCH" : (r.correct == 1 ? " ok" : ""));
    }
    return failures ? 1 : 0;
}

int usage() {
    std::fprintf(stderr,
                 "usage: convbench --csv OPS.csv --out RESULTS.csv [--datagen random|constant]\n"
                 "                 [--exec main|baseline|correctness] [--warmups W] [--runs R] [--seed S]\n"
                 "                 [--dry-run] [--dump DIR]\n");
    return 2;
}

}  // namespace

int main(int argc, char** argv) {
    std::string csv, out, datagen = "random", exec = "main", dump;
    int warmups = 10, runs = 100;
    uint64_t seed = 1000;
    bool dry = false;
    for (int i = 1; i < argc; ++i) {
        const std::string a = argv[i];
        auto val = [&]() -> std::string { return i + 1 < argc ? std::string(argv[++i]) : std::string(); };
        if (a == "--csv") csv = val();
        else if (a == "--out") out = val();
        else if (a == "--datagen") datagen = val();
        else if (a == "--exec") exec = val();
        else if (a == "--warmups") warmups = std::atoi(val().c_str());
        else if (a == "--runs") runs = std::atoi(val().c_str());
        else if (a == "--seed") seed = std::strtoull(val().c_str(), nullptr, 10);
        else if (a == "--dry-run") dry = true;
        else if (a == "--dump") dump = val();
        else return usage();
    }
    if (csv.empty() || out.empty() || (datagen != "random" && datagen != "constant") ||
        (exec != "main" && exec != "baseline" && exec != "correctness") || warmups < 0 || runs < 1)
        return usage();
    std::vector<Op> ops;
    std::string err;
    if (!read_ops(csv, &ops, &err)) {
        std::fprintf(stderr, "convbench: %s: %s\n", csv.c_str(), err.c_str());
        return 2;
    }
    Conv2dBench bench;
    return bench.convset_exec(ops, datagen, exec, warmups, runs, seed, dry, out, dump);
}

// frontend.cpp -- the program front end of libdsim: programs written op by op
// as text, interpreted over a mixed abstract/concrete domain and lowered to
// the explicit op-table format of dsim_simulate_tables (include/dsim.h).
// Host code only: no HIP call, no device memory, nothing kept between calls.
//
// Interpretation (Sec. 3, Algorithm 1).  The ops are stepped through in
// program order over a state that maps every variable to a value; each op
// type is evaluated by the implementation that matches the kinds of its
// arguments.  A value is concrete -- an int64 or fp64 array of any rank,
// rank 0 being a number -- or abstract: a tensor (element type, shape or
// unknown, device) or a scalar (element type, device or none).  Op types
// carry concrete, mixed and abstract implementations and the most precise
// one that matches is taken (Sec. 3.3, the Reshape snippet of Fig. 4): an op
// whose arguments are all concrete is evaluated here; Shape of a tensor of
// known shape is concrete; Reshape of a tensor by a concrete target has a
// known shape; everything else is computed on types.  The abstract-only
// interpretation replaces every concrete value by its type as soon as it
// appears (shape arithmetic is typed Int32, fp64 values Float64).
//
// Lowering (the simulator of Sec. 3.3 on the table format).  Always on the
// mixed interpretation.  An op that yields no abstract tensor runs on the
// host and emits nothing; a view (Reshape, Unsqueeze, Squeeze, Flatten,
// Identity) shares its input's memory and emits nothing; every other op on
// abstract tensors is one record: compute on the one device of its tensors
// (matrix products cost class 1), Send (source -> destination), AllReduce
// (in place over the devices of its inputs).  Memory is per storage: the
// tensors an op creates get one each, allocated by its record on its device
// (a Send's receiver); a storage is freed by the last record that reads it
// (or creates it, if nothing reads it); parameters are resident from t = 0,
// those marked keep for good; a storage last read by an AllReduce stays
// live (the collective works in place and frees nothing).  Costs: compute
// bytes are the sizes of every abstract input and output tensor; flops are 1
// per output element for the elementwise ops (Gelu 8, Softmax 5,
// LayerNormalization 8, Cast 0), 2 * (output elements) * k for MatMul and
// Gemm (plus one per output element for Gemm's bias), none for Transpose,
// Concat, Split and Gather; Send and AllReduce move their (first) input's
// bytes.  A matrix product's record also carries its reduction length k
// (MatMul: the left operand's last dimension; Gemm: the shared dimension),
// which the empirical MatMul cost reads.
#include <algorithm>
#include <cerrno>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <string_view>
#include <thread>
#include <unordered_map>
#include <vector>

#include "internal.h"

namespace dsim {
namespace {

using u128 = unsigned __int128;

constexpr int kMaxRank = 16;
constexpr int64_t kMaxConcrete = (int64_t)1 << 20;   // elements of one concrete value
constexpr int kMaxOut = 4096;                         // results of one op
constexpr int kMaxNest = 32;                          // nesting depth of a literal

// ---------------------------------------------------------------------------
// Errors: raised as a C++ exception inside this file, turned into a
// dsim_status at the C boundary.
// ---------------------------------------------------------------------------
struct Failure {
    dsim_status st;
    char msg[440];
};

[[noreturn]] __attribute__((format(printf, 2, 3))) void throw_fail(dsim_status st, const char *fmt, ...)
{
    Failure f;
    f.st = st;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(f.msg, sizeof f.msg, fmt, ap);
    va_end(ap);
    throw f;
}

// ---------------------------------------------------------------------------
// Element types
// ---------------------------------------------------------------------------
enum DType : int8_t { F64, F32, F16, BF16, I64, I32, I8, BOOL, N_DTYPE };
const char *const kDtName[N_DTYPE] = {"Float64", "Float32", "Float16", "BFloat16", "Int64", "Int32", "Int8", "Bool"};
const int kDtSize[N_DTYPE] = {8, 4, 2, 2, 8, 4, 1, 1};

int dtype_of(std::string_view s)
{
    for (int i = 0; i < N_DTYPE; ++i)
        if (s == kDtName[i]) return i;
    return -1;
}

// ---------------------------------------------------------------------------
// Shapes and values
// ---------------------------------------------------------------------------
struct Shape {
    int32_t rank = 0;
    int64_t d[kMaxRank];
    void push(int64_t v)
    {
        if (rank == kMaxRank) throw_fail(DSIM_ERANGE, "a shape of rank above %d", kMaxRank);
        d[rank++] = v;
    }
    bool operator==(const Shape &o) const
    {
        if (rank != o.rank) return false;
        for (int i = 0; i < rank; ++i)
            if (d[i] != o.d[i]) return false;
        return true;
    }
};

// product of d[lo..hi), every dimension >= 0; beyond 2^63 - 1 is an error
int64_t prod(const Shape &s, int lo, int hi)
{
    int64_t n = 1;
    for (int i = lo; i < hi; ++i)
        if (__builtin_mul_overflow(n, s.d[i], &n)) throw_fail(DSIM_ERANGE, "a tensor of 2^63 elements or more");
    return n;
}
int64_t numel(const Shape &s) { return prod(s, 0, s.rank); }

std::string show_shape(const Shape &s, bool tuple = true)
{
    std::string o(tuple ? "(" : "[");
    char b[24];
    for (int i = 0; i < s.rank; ++i) {
        snprintf(b, sizeof b, "%s%lld", i ? ", " : "", (long long)s.d[i]);
        o += b;
    }
    if (tuple && s.rank == 1) o += ",";
    o += tuple ? ")" : "]";
    return o;
}

enum Kind : int8_t { CONC, TENSOR, SCALAR };

struct Value {
    Kind kind = CONC;
    int8_t dt = I64;      // concrete: I64 or F64; abstract: the element type
    bool known = true;    // tensor: the shape is known
    int32_t dev = -1;     // abstract: device, -1 = none
    Shape shape;          // concrete: the array's shape; tensor: its shape when known
    std::vector<int64_t> iv;
    std::vector<double> fv;

    bool flt() const { return dt == F64; }
    double at(int64_t i) const { return dt == F64 ? fv[i] : (double)iv[i]; }
};

bool is_c(const Value &v) { return v.kind == CONC; }
bool is_t(const Value &v) { return v.kind == TENSOR; }
bool is_s(const Value &v) { return v.kind == SCALAR; }

Value tensor(int dt, const Shape *shape, int dev)
{
    Value v;
    v.kind = TENSOR;
    v.dt = (int8_t)dt;
    v.dev = dev;
    v.known = shape != nullptr;
    if (shape) v.shape = *shape;
    return v;
}

Value scalar(int dt, int dev)
{
    Value v;
    v.kind = SCALAR;
    v.dt = (int8_t)dt;
    v.dev = dev;
    return v;
}

Value conc(bool flt, const Shape &shape)
{
    Value v;
    v.kind = CONC;
    v.dt = flt ? F64 : I64;
    v.shape = shape;
    int64_t n = numel(shape);
    if (n > kMaxConcrete) throw_fail(DSIM_ERANGE, "a concrete value of more than 2^20 elements");
    if (flt)
        v.fv.assign((size_t)n, 0.0);
    else
        v.iv.assign((size_t)n, 0);
    return v;
}

// The type of a concrete value on device dev (abstract values unchanged):
// fp64 arrays are Float64, integer shape arithmetic Int32.
Value abstract_of(const Value &v, int dev)
{
    if (!is_c(v)) return v;
    int dt = v.flt() ? F64 : I32;
    if (v.shape.rank == 0) return scalar(dt, dev);
    return tensor(dt, &v.shape, dev);
}

// the one device of the abstract values among args, -1 if none
int device_of(const Value *const *a, int n)
{
    int dev = -1;
    for (int i = 0; i < n; ++i) {
        if (is_c(*a[i]) || a[i]->dev < 0) continue;
        if (dev >= 0 && a[i]->dev != dev)
            throw_fail(DSIM_EINVAL, "inputs on different devices [%d, %d]", std::min(dev, a[i]->dev),
                  std::max(dev, a[i]->dev));
        dev = a[i]->dev;
    }
    return dev;
}

// ---------------------------------------------------------------------------
// Literals (attribute values, concrete inputs)
// ---------------------------------------------------------------------------
struct Lit {
    enum T : int8_t { INT, FLT, STR, LIST } t = INT;
    int64_t i = 0;
    double f = 0.0;
    std::string_view s;
    std::vector<Lit> items;
};

bool is_space(char c) { return c == ' ' || c == '\t' || c == '\r' || c == '\n' || c == '\f' || c == '\v'; }
bool is_word(char c) { return (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z') || (c >= '0' && c <= '9') || c == '_'; }

void skip_ws(std::string_view s, size_t &p)
{
    while (p < s.size() && is_space(s[p])) ++p;
}

std::string_view trim(std::string_view s)
{
    size_t a = 0, b = s.size();
    while (a < b && is_space(s[a])) ++a;
    while (b > a && is_space(s[b - 1])) --b;
    return s.substr(a, b - a);
}

Lit parse_lit(std::string_view s, size_t &p, int depth)
{
    if (depth > kMaxNest) throw_fail(DSIM_EINVAL, "a literal nested more than %d deep", kMaxNest);
    skip_ws(s, p);
    if (p >= s.size()) throw_fail(DSIM_EINVAL, "a value is missing");
    Lit l;
    char c = s[p];
    if (c == '[' || c == '(') {
        char close = c == '[' ? ']' : ')';
        l.t = Lit::LIST;
        ++p;
        skip_ws(s, p);
        if (p < s.size() && s[p] == close) {
            ++p;
            return l;
        }
        for (;;) {
            l.items.push_back(parse_lit(s, p, depth + 1));
            skip_ws(s, p);
            if (p >= s.size()) throw_fail(DSIM_EINVAL, "an unclosed list");
            if (s[p] == ',') {
                ++p;
                skip_ws(s, p);
                if (p < s.size() && s[p] == close) {
                    ++p;
                    break;
                }
                continue;
            }
            if (s[p] == close) {
                ++p;
                break;
            }
            throw_fail(DSIM_EINVAL, "unexpected '%c' in a list", s[p]);
        }
        return l;
    }
    if (c == '"' || c == '\'') {
        size_t q = s.find(c, p + 1);
        if (q == std::string_view::npos) throw_fail(DSIM_EINVAL, "an unclosed string");
        l.t = Lit::STR;
        l.s = s.substr(p + 1, q - p - 1);
        p = q + 1;
        return l;
    }
    size_t q = p;
    while (q < s.size() && (is_word(s[q]) || s[q] == '+' || s[q] == '-' || s[q] == '.')) ++q;
    std::string tok(s.substr(p, q - p));
    p = q;
    if (tok.empty()) throw_fail(DSIM_EINVAL, "unexpected '%c' in a value", c);
    if (tok == "True" || tok == "true" || tok == "False" || tok == "false") {
        l.t = Lit::INT;
        l.i = tok[0] == 'T' || tok[0] == 't';
        return l;
    }
    const double inf = INFINITY;
    if (tok == "inf" || tok == "+inf" || tok == "Infinity" || tok == "+Infinity" || tok == "-inf" ||
        tok == "-Infinity" || tok == "nan" || tok == "NaN") {
        l.t = Lit::FLT;
        l.f = tok[0] == 'n' || tok[0] == 'N' ? NAN : (tok[0] == '-' ? -inf : inf);
        return l;
    }
    for (char ch : tok)
        if (!((ch >= '0' && ch <= '9') || ch == '+' || ch == '-' || ch == '.' || ch == 'e' || ch == 'E'))
            throw_fail(DSIM_EINVAL, "cannot read '%s' as a number", tok.c_str());
    char *end = nullptr;
    if (tok.find_first_of(".eE") == std::string::npos) {
        errno = 0;
        long long v = strtoll(tok.c_str(), &end, 10);
        if (*end == 0) {
            if (errno == ERANGE) throw_fail(DSIM_ERANGE, "the integer %s is beyond 64 bits", tok.c_str());
            l.t = Lit::INT;
            l.i = v;
            return l;
        }
    }
    double v = strtod(tok.c_str(), &end);
    if (*end != 0) throw_fail(DSIM_EINVAL, "cannot read '%s' as a number", tok.c_str());
    l.t = Lit::FLT;
    l.f = v;
    return l;
}

Lit parse_lit_all(std::string_view s)
{
    size_t p = 0;
    Lit l = parse_lit(s, p, 0);
    skip_ws(s, p);
    if (p != s.size()) throw_fail(DSIM_EINVAL, "unexpected text after a value");
    return l;
}

bool lit_has_float(const Lit &l)
{
    if (l.t == Lit::FLT) return true;
    if (l.t == Lit::STR) throw_fail(DSIM_EINVAL, "a string where a number is expected");
    if (l.t == Lit::LIST)
        for (const Lit &x : l.items)
            if (lit_has_float(x)) return true;
    return false;
}

void lit_fill(const Lit &l, const Shape &sh, int dim, Value &v, int64_t &k)
{
    if (dim == sh.rank) {
        if (l.t == Lit::LIST) throw_fail(DSIM_EINVAL, "a ragged list");
        if (v.flt())
            v.fv[(size_t)k++] = l.t == Lit::FLT ? l.f : (double)l.i;
        else
            v.iv[(size_t)k++] = l.i;
        return;
    }
    if (l.t != Lit::LIST || (int64_t)l.items.size() != sh.d[dim]) throw_fail(DSIM_EINVAL, "a ragged list");
    for (const Lit &x : l.items) lit_fill(x, sh, dim + 1, v, k);
}

// a number or a rectangular nested list as a concrete value (int64 unless
// some element is a float)
Value lit_value(const Lit &l)
{
    Shape sh;
    for (const Lit *x = &l; x->t == Lit::LIST;) {
        sh.push((int64_t)x->items.size());
        if (x->items.empty()) break;
        x = &x->items[0];
    }
    bool flt = lit_has_float(l) || (sh.rank > 0 && numel(sh) == 0);
    Value v = conc(flt, sh);
    int64_t k = 0;
    lit_fill(l, sh, 0, v, k);
    return v;
}

// ---------------------------------------------------------------------------
// Attributes
// ---------------------------------------------------------------------------
struct Attr {
    std::string_view key;
    Lit val;
};

struct Attrs {
    std::vector<Attr> a;
    const Lit *find(const char *key) const
    {
        for (const Attr &x : a)
            if (x.key == key) return &x.val;
        return nullptr;
    }
    int64_t get_int(const char *key, int64_t dflt, bool required = false) const
    {
        const Lit *l = find(key);
        if (!l) {
            if (required) throw_fail(DSIM_EINVAL, "attribute %s is missing", key);
            return dflt;
        }
        if (l->t != Lit::INT) throw_fail(DSIM_EINVAL, "attribute %s must be an integer", key);
        return l->i;
    }
    // a flat integer list; false if absent (and not required)
    bool get_ints(const char *key, std::vector<int64_t> &out, bool required) const
    {
        out.clear();
        const Lit *l = find(key);
        if (!l) {
            if (required) throw_fail(DSIM_EINVAL, "attribute %s is missing", key);
            return false;
        }
        if (l->t != Lit::LIST) throw_fail(DSIM_EINVAL, "attribute %s must be a list of integers", key);
        for (const Lit &x : l->items) {
            if (x.t != Lit::INT) throw_fail(DSIM_EINVAL, "attribute %s must be a list of integers", key);
            out.push_back(x.i);
        }
        return true;
    }
};

// ---------------------------------------------------------------------------
// Op types
// ---------------------------------------------------------------------------
enum OpT : int8_t {
    O_CONSTANT, O_SHAPE, O_GATHER, O_UNSQUEEZE, O_SQUEEZE, O_CONCAT, O_RESHAPE, O_ADD, O_SUB, O_MUL, O_DIV,
    O_POW, O_RELU, O_NEG, O_SQRT, O_EXP, O_TANH, O_ERF, O_GELU, O_IDENTITY, O_CAST, O_SOFTMAX, O_LAYERNORM,
    O_TRANSPOSE, O_FLATTEN, O_SPLIT, O_MATMUL, O_GEMM, O_SEND, O_ALLREDUCE, N_OPT
};
const char *const kOpName[N_OPT] = {
    "Constant", "Shape", "Gather", "Unsqueeze", "Squeeze", "Concat", "Reshape", "Add", "Sub", "Mul", "Div",
    "Pow", "Relu", "Neg", "Sqrt", "Exp", "Tanh", "Erf", "Gelu", "Identity", "Cast", "Softmax",
    "LayerNormalization", "Transpose", "Flatten", "Split", "MatMul", "Gemm", "Send", "AllReduce"};
// flops per output element of the elementwise ops, -1 for the others
const int kEltFlops[N_OPT] = {-1, -1, -1, -1, -1, -1, -1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 8, -1, 0, 5, 8,
                              -1, -1, -1, -1, -1, -1, -1};

int op_of(std::string_view s)
{
    for (int i = 0; i < N_OPT; ++i)
        if (s == kOpName[i]) return i;
    return -1;
}

bool is_view(int op)
{
    return op == O_RESHAPE || op == O_UNSQUEEZE || op == O_SQUEEZE || op == O_FLATTEN || op == O_IDENTITY;
}

[[noreturn]] void no_impl(int op, std::string_view name, const Value *const *a, int n)
{
    std::string kinds;
    for (int i = 0; i < n; ++i) {
        if (i) kinds += ", ";
        kinds += is_c(*a[i]) ? "concrete" : is_t(*a[i]) ? "Tensor" : "Scalar";
    }
    throw_fail(DSIM_EINVAL, "no implementation of %.*s for arguments [%s]", (int)name.size(), name.data(),
          kinds.c_str());
    (void)op;
}

// ---------------------------------------------------------------------------
// Shape helpers
// ---------------------------------------------------------------------------
int norm_axis(int64_t ax, int rank, const char *what)
{
    int64_t a = ax < 0 ? ax + rank : ax;
    if (a < 0 || a >= rank) throw_fail(DSIM_EINVAL, "%s axis %lld out of range for rank %d", what, (long long)ax, rank);
    return (int)a;
}

Shape bcast(const Shape &a, const Shape &b)
{
    Shape r;
    int n = std::max(a.rank, b.rank);
    r.rank = n;
    for (int i = 0; i < n; ++i) {
        int64_t x = i < n - a.rank ? 1 : a.d[i - (n - a.rank)];
        int64_t y = i < n - b.rank ? 1 : b.d[i - (n - b.rank)];
        if (x != y && x != 1 && y != 1)
            throw_fail(DSIM_EINVAL, "shapes %s and %s cannot be broadcast", show_shape(a).c_str(), show_shape(b).c_str());
        r.d[i] = x == 1 ? y : x;
    }
    return r;
}

Shape unsq_shape(const Shape &s, const std::vector<int64_t> &axes)
{
    int out = s.rank + (int)axes.size();
    if (out > kMaxRank) throw_fail(DSIM_ERANGE, "a shape of rank above %d", kMaxRank);
    bool ins[kMaxRank] = {};
    for (int64_t a : axes) {
        int k = norm_axis(a, out, "Unsqueeze");
        if (ins[k]) throw_fail(DSIM_EINVAL, "Unsqueeze axis %lld repeated", (long long)a);
        ins[k] = true;
    }
    Shape r;
    for (int i = 0, j = 0; i < out; ++i) r.push(ins[i] ? 1 : s.d[j++]);
    return r;
}

Shape squeeze_shape(const Shape &s, const std::vector<int64_t> &axes, bool all)
{
    bool drop[kMaxRank] = {};
    if (all) {
        for (int i = 0; i < s.rank; ++i) drop[i] = s.d[i] == 1;
    } else {
        for (int64_t a : axes) {
            int k = norm_axis(a, s.rank, "Squeeze");
            if (drop[k]) throw_fail(DSIM_EINVAL, "Squeeze axis %lld repeated", (long long)a);
            if (s.d[k] != 1)
                throw_fail(DSIM_EINVAL, "cannot squeeze dimension %d of size %lld", k, (long long)s.d[k]);
            drop[k] = true;
        }
    }
    Shape r;
    for (int i = 0; i < s.rank; ++i)
        if (!drop[i]) r.push(s.d[i]);
    return r;
}

// Reshape's target: 0 copies the input's dimension, one -1 is inferred
Shape reshape_target(const Shape &s, const Value &t)
{
    if (t.flt() || t.shape.rank != 1) throw_fail(DSIM_EINVAL, "a Reshape target must be a list of integers");
    Shape r;
    int infer = -1;
    for (int64_t i = 0; i < t.shape.d[0]; ++i) {
        int64_t v = t.iv[(size_t)i];
        if (v == 0) {
            if (i >= s.rank) throw_fail(DSIM_EINVAL, "Reshape copies dimension %lld of a rank-%d tensor", (long long)i, s.rank);
            v = s.d[i];
        } else if (v == -1) {
            if (infer >= 0) throw_fail(DSIM_EINVAL, "a Reshape target with more than one -1");
            infer = (int)i;
            v = 1;
        } else if (v < 0) {
            throw_fail(DSIM_EINVAL, "a Reshape target entry %lld", (long long)v);
        }
        r.push(v);
    }
    int64_t total = numel(s), known = numel(r);
    if (infer >= 0) {
        if (known == 0 || total % known != 0)
            throw_fail(DSIM_EINVAL, "cannot reshape %s to %s", show_shape(s).c_str(),
                  show_shape(r, false).c_str());
        r.d[infer] = total / known;
    }
    if (numel(r) != total) {
        Shape tt;
        for (int64_t i = 0; i < t.shape.d[0]; ++i) tt.push(t.iv[(size_t)i]);
        throw_fail(DSIM_EINVAL, "cannot reshape %s to %s", show_shape(s).c_str(), show_shape(tt, false).c_str());
    }
    return r;
}

// ---------------------------------------------------------------------------
// Concrete arithmetic (numpy's rules for int64 / fp64 arrays: integer
// results wrap, division is true division)
// ---------------------------------------------------------------------------
int64_t wrap_add(int64_t a, int64_t b) { return (int64_t)((uint64_t)a + (uint64_t)b); }
int64_t wrap_sub(int64_t a, int64_t b) { return (int64_t)((uint64_t)a - (uint64_t)b); }
int64_t wrap_mul(int64_t a, int64_t b) { return (int64_t)((uint64_t)a * (uint64_t)b); }
int64_t wrap_pow(int64_t a, int64_t e)
{
    uint64_t r = 1, x = (uint64_t)a;
    for (uint64_t k = (uint64_t)e; k; k >>= 1) {
        if (k & 1) r *= x;
        x *= x;
    }
    return (int64_t)r;
}

Value binary_c(int op, const Value &a, const Value &b)
{
    Shape r = bcast(a.shape, b.shape);
    bool flt = op == O_DIV || a.flt() || b.flt();
    Value v = conc(flt, r);
    int64_t n = numel(r);
    // element strides of a and b in r's index space (0 on broadcast axes)
    int64_t sa[kMaxRank], sb[kMaxRank];
    int64_t ka = 1, kb = 1;
    for (int i = r.rank - 1; i >= 0; --i) {
        int ia = i - (r.rank - a.shape.rank), ib = i - (r.rank - b.shape.rank);
        int64_t da = ia >= 0 ? a.shape.d[ia] : 1, db = ib >= 0 ? b.shape.d[ib] : 1;
        sa[i] = da == 1 ? 0 : ka;
        sb[i] = db == 1 ? 0 : kb;
        ka *= da;
        kb *= db;
    }
    int64_t idx[kMaxRank] = {};
    int64_t pa = 0, pb = 0;
    for (int64_t k = 0; k < n; ++k) {
        if (flt) {
            double x = a.at(pa), y = b.at(pb), z;
            switch (op) {
            case O_ADD: z = x + y; break;
            case O_SUB: z = x - y; break;
            case O_MUL: z = x * y; break;
            case O_DIV: z = x / y; break;
            default: z = std::pow(x, y); break;
            }
            v.fv[(size_t)k] = z;
        } else {
            int64_t x = a.iv[(size_t)pa], y = b.iv[(size_t)pb], z;
            switch (op) {
            case O_ADD: z = wrap_add(x, y); break;
            case O_SUB: z = wrap_sub(x, y); break;
            case O_MUL: z = wrap_mul(x, y); break;
            default:
                if (y < 0) throw_fail(DSIM_EINVAL, "integers to negative integer powers are not allowed");
                z = wrap_pow(x, y);
                break;
            }
            v.iv[(size_t)k] = z;
        }
        for (int i = r.rank - 1; i >= 0; --i) {   // next index of r
            pa += sa[i];
            pb += sb[i];
            if (++idx[i] < r.d[i]) break;
            pa -= sa[i] * r.d[i];
            pb -= sb[i] * r.d[i];
            idx[i] = 0;
        }
    }
    return v;
}

Value unary_c(int op, const Value &a)
{
    bool flt = a.flt() || op == O_SQRT || op == O_EXP || op == O_TANH;
    Value v = conc(flt, a.shape);
    int64_t n = numel(a.shape);
    for (int64_t k = 0; k < n; ++k) {
        if (!flt) {
            int64_t x = a.iv[(size_t)k];
            v.iv[(size_t)k] = op == O_RELU ? std::max<int64_t>(x, 0) : op == O_NEG ? wrap_sub(0, x) : x;
        } else {
            double x = a.at(k);
            switch (op) {
            case O_RELU: v.fv[(size_t)k] = x < 0.0 ? 0.0 : x; break;
            case O_NEG: v.fv[(size_t)k] = -x; break;
            case O_SQRT: v.fv[(size_t)k] = std::sqrt(x); break;
            case O_EXP: v.fv[(size_t)k] = std::exp(x); break;
            case O_TANH: v.fv[(size_t)k] = std::tanh(x); break;
            default: v.fv[(size_t)k] = x; break;
            }
        }
    }
    return v;
}

// the index of one Gather entry along an axis of n entries
int64_t gather_index(int64_t i, int64_t n)
{
    int64_t j = i < 0 ? i + n : i;
    if (j < 0 || j >= n) throw_fail(DSIM_EINVAL, "index %lld out of range for a dimension of %lld", (long long)i, (long long)n);
    return j;
}

// ---------------------------------------------------------------------------
// One op: its results from its arguments (the most precise implementation)
// ---------------------------------------------------------------------------
std::string show_list(const std::vector<int64_t> &v)
{
    std::string o("[");
    char b[24];
    for (size_t i = 0; i < v.size(); ++i) {
        snprintf(b, sizeof b, "%s%lld", i ? ", " : "", (long long)v[i]);
        o += b;
    }
    return o + "]";
}

struct Evaluator {
    std::vector<int64_t> ints;   // scratch for integer-list attributes

    void run(int op, std::string_view name, const Attrs &at, const Value *const *a, int n, std::vector<Value> &out)
    {
        out.clear();
        switch (op) {
        case O_CONSTANT: {
            if (n != 0) no_impl(op, name, a, n);
            const Lit *l = at.find("value");
            if (!l) throw_fail(DSIM_EINVAL, "attribute value is missing");
            out.push_back(lit_value(*l));
            return;
        }
        case O_SHAPE: {
            if (n != 1 || is_s(*a[0])) no_impl(op, name, a, n);
            const Value &x = *a[0];
            if (is_t(x) && !x.known) {
                out.push_back(tensor(I32, nullptr, x.dev));
                return;
            }
            Shape s;
            s.push(x.shape.rank);
            Value v = conc(false, s);
            for (int i = 0; i < x.shape.rank; ++i) v.iv[(size_t)i] = x.shape.d[i];
            out.push_back(std::move(v));
            return;
        }
        case O_GATHER: {
            if (n != 2) no_impl(op, name, a, n);
            const Value &d = *a[0], &ix = *a[1];
            int64_t ax = at.get_int("axis", 0);
            if (is_c(d) && is_c(ix)) {
                if (ix.flt()) throw_fail(DSIM_EINVAL, "Gather indices must be integers");
                if (d.shape.rank == 0) throw_fail(DSIM_EINVAL, "Gather from a number");
                int k = norm_axis(ax, d.shape.rank, "Gather");
                Shape r;
                for (int i = 0; i < k; ++i) r.push(d.shape.d[i]);
                for (int i = 0; i < ix.shape.rank; ++i) r.push(ix.shape.d[i]);
                for (int i = k + 1; i < d.shape.rank; ++i) r.push(d.shape.d[i]);
                Value v = conc(d.flt(), r);
                int64_t outer = prod(d.shape, 0, k), inner = prod(d.shape, k + 1, d.shape.rank);
                int64_t len = d.shape.d[k], ni = numel(ix.shape), o = 0;
                for (int64_t p = 0; p < outer; ++p)
                    for (int64_t q = 0; q < ni; ++q) {
                        int64_t j = gather_index(ix.iv[(size_t)q], len);
                        for (int64_t w = 0; w < inner; ++w, ++o) {
                            int64_t src = (p * len + j) * inner + w;
                            if (v.flt())
                                v.fv[(size_t)o] = d.fv[(size_t)src];
                            else
                                v.iv[(size_t)o] = d.iv[(size_t)src];
                        }
                    }
                out.push_back(std::move(v));
                return;
            }
            if (!is_t(d)) no_impl(op, name, a, n);
            if (is_c(ix) && ix.flt()) throw_fail(DSIM_EINVAL, "Gather indices must be integers");
            int dev = device_of(a, 2);
            if (d.known && d.shape.rank == 1 && (is_s(ix) || (is_c(ix) && ix.shape.rank == 0))) {
                out.push_back(scalar(d.dt, dev));
                return;
            }
            bool iknown = is_s(ix) || is_c(ix) || ix.known;
            if (!d.known || !iknown) {
                out.push_back(tensor(d.dt, nullptr, dev));
                return;
            }
            Shape is;
            if (!is_s(ix)) is = ix.shape;
            int k = norm_axis(ax, d.shape.rank, "Gather");
            Shape r;
            for (int i = 0; i < k; ++i) r.push(d.shape.d[i]);
            for (int i = 0; i < is.rank; ++i) r.push(is.d[i]);
            for (int i = k + 1; i < d.shape.rank; ++i) r.push(d.shape.d[i]);
            out.push_back(tensor(d.dt, &r, dev));
            return;
        }
        case O_UNSQUEEZE: {
            if (n != 1) no_impl(op, name, a, n);
            at.get_ints("axes", ints, true);
            const Value &x = *a[0];
            if (is_c(x)) {
                Value v = x;
                v.shape = unsq_shape(x.shape, ints);
                out.push_back(std::move(v));
            } else if (is_s(x)) {
                Shape s0;
                Shape r = unsq_shape(s0, ints);
                out.push_back(tensor(x.dt, &r, x.dev));
            } else if (!x.known) {
                out.push_back(x);
            } else {
                Shape r = unsq_shape(x.shape, ints);
                out.push_back(tensor(x.dt, &r, x.dev));
            }
            return;
        }
        case O_SQUEEZE: {
            if (n != 1 || is_s(*a[0])) no_impl(op, name, a, n);
            bool all = !at.get_ints("axes", ints, false);
            const Value &x = *a[0];
            Value v = x;
            if (is_c(x) || x.known) v.shape = squeeze_shape(x.shape, ints, all);
            out.push_back(std::move(v));
            return;
        }
        case O_CONCAT: {
            if (n < 1) throw_fail(DSIM_EINVAL, "Concat of no values");
            int64_t ax = at.get_int("axis", 0);
            bool allc = true, flt = false;
            for (int i = 0; i < n; ++i) {
                allc = allc && is_c(*a[i]);
                flt = flt || (is_c(*a[i]) && a[i]->flt());
            }
            if (allc) {
                // numpy's atleast_1d: numbers are rank-1 lists of one entry
                Shape s0 = a[0]->shape;
                if (s0.rank == 0) s0.push(1);
                int k = norm_axis(ax, s0.rank, "Concat");
                int64_t total = 0;
                for (int i = 0; i < n; ++i) {
                    Shape si = a[i]->shape;
                    if (si.rank == 0) si.push(1);
                    if (si.rank != s0.rank) throw_fail(DSIM_EINVAL, "Concat of values of different ranks");
                    for (int j = 0; j < si.rank; ++j)
                        if (j != k && si.d[j] != s0.d[j]) throw_fail(DSIM_EINVAL, "Concat of mismatched shapes");
                    total += si.d[k];
                }
                Shape r = s0;
                r.d[k] = total;
                Value v = conc(flt, r);
                int64_t outer = prod(s0, 0, k), inner = prod(s0, k + 1, s0.rank), o = 0;
                for (int64_t p = 0; p < outer; ++p)
                    for (int i = 0; i < n; ++i) {
                        int64_t w = (a[i]->shape.rank == 0 ? 1 : a[i]->shape.d[k]) * inner;
                        for (int64_t q = 0; q < w; ++q, ++o) {
                            int64_t src = p * w + q;
                            if (flt)
                                v.fv[(size_t)o] = a[i]->at(src);
                            else
                                v.iv[(size_t)o] = a[i]->iv[(size_t)src];
                        }
                    }
                out.push_back(std::move(v));
                return;
            }
            std::vector<Value> av;
            av.reserve((size_t)n);
            std::vector<const Value *> ap;
            for (int i = 0; i < n; ++i) av.push_back(abstract_of(*a[i], -1));
            for (const Value &x : av) ap.push_back(&x);
            int dev = device_of(ap.data(), n);
            bool unknown = false;
            for (const Value &x : av) unknown = unknown || is_s(x) || !x.known;
            if (unknown) {
                out.push_back(tensor(av[0].dt, nullptr, dev));
                return;
            }
            Shape r = av[0].shape;
            int k = norm_axis(ax, r.rank, "Concat");
            int64_t total = 0;
            for (const Value &x : av) {
                if (x.shape.rank != r.rank) throw_fail(DSIM_EINVAL, "Concat of values of different ranks");
                for (int j = 0; j < r.rank; ++j)
                    if (j != k && x.shape.d[j] != r.d[j]) throw_fail(DSIM_EINVAL, "Concat of mismatched shapes");
                if (__builtin_add_overflow(total, x.shape.d[k], &total))
                    throw_fail(DSIM_ERANGE, "a tensor of 2^63 elements or more");
            }
            r.d[k] = total;
            out.push_back(tensor(av[0].dt, &r, dev));
            return;
        }
        case O_RESHAPE: {
            if (n != 2) no_impl(op, name, a, n);
            const Value &x = *a[0], &t = *a[1];
            if (is_c(x) && is_c(t)) {
                Value v = x;
                v.shape = reshape_target(x.shape, t);
                out.push_back(std::move(v));
            } else if (is_t(x) && is_c(t)) {
                if (x.known) {
                    Shape r = reshape_target(x.shape, t);
                    out.push_back(tensor(x.dt, &r, x.dev));
                } else {
                    out.push_back(tensor(x.dt, nullptr, x.dev));
                }
            } else if (is_t(x) && !is_c(t)) {
                out.push_back(tensor(x.dt, nullptr, x.dev));   // the target is not known
            } else {
                no_impl(op, name, a, n);
            }
            return;
        }
        case O_ADD: case O_SUB: case O_MUL: case O_DIV: case O_POW: {
            if (n != 2) no_impl(op, name, a, n);
            if (is_c(*a[0]) && is_c(*a[1])) {
                out.push_back(binary_c(op, *a[0], *a[1]));
                return;
            }
            Value va = abstract_of(*a[0], -1), vb = abstract_of(*a[1], -1);
            const Value *ab[2] = {&va, &vb};
            int dev = device_of(ab, 2);
            if (is_s(va) && is_s(vb)) {
                out.push_back(scalar(va.dt, dev));
                return;
            }
            int dt = is_t(va) ? va.dt : vb.dt;
            if ((is_t(va) && !va.known) || (is_t(vb) && !vb.known)) {
                out.push_back(tensor(dt, nullptr, dev));
                return;
            }
            Shape r = bcast(is_s(va) ? Shape() : va.shape, is_s(vb) ? Shape() : vb.shape);
            out.push_back(tensor(dt, &r, dev));
            return;
        }
        case O_RELU: case O_NEG: case O_SQRT: case O_EXP: case O_TANH: case O_ERF: case O_GELU: case O_IDENTITY: {
            if (n != 1) no_impl(op, name, a, n);
            if (is_c(*a[0])) {
                if (op == O_ERF || op == O_GELU) no_impl(op, name, a, n);
                out.push_back(unary_c(op, *a[0]));
            } else {
                out.push_back(*a[0]);
            }
            return;
        }
        case O_CAST: {
            if (n != 1) no_impl(op, name, a, n);
            const Lit *to = at.find("to");
            if (!to || to->t != Lit::STR) throw_fail(DSIM_EINVAL, "attribute to must be an element type name");
            int dt = dtype_of(to->s);
            if (dt < 0) throw_fail(DSIM_EINVAL, "unknown element type %.*s", (int)to->s.size(), to->s.data());
            const Value &x = *a[0];
            if (is_c(x)) {
                bool flt = dt == F64 || dt == F32 || dt == F16 || dt == BF16;
                Value v = conc(flt, x.shape);
                int64_t m = numel(x.shape);
                for (int64_t k = 0; k < m; ++k) {
                    if (flt) {
                        v.fv[(size_t)k] = x.at(k);
                    } else if (!x.flt()) {
                        v.iv[(size_t)k] = x.iv[(size_t)k];
                    } else {
                        double f = x.fv[(size_t)k];
                        if (!(f > -9223372036854775808.0 - 1.0 && f < 9223372036854775808.0))
                            throw_fail(DSIM_EINVAL, "cannot cast %g to an integer", f);
                        v.iv[(size_t)k] = (int64_t)f;
                    }
                }
                out.push_back(std::move(v));
            } else if (is_s(x)) {
                out.push_back(scalar(dt, x.dev));
            } else {
                Value v = x;
                v.dt = (int8_t)dt;
                out.push_back(std::move(v));
            }
            return;
        }
        case O_SOFTMAX:
            if (n != 1 || !is_t(*a[0])) no_impl(op, name, a, n);
            out.push_back(*a[0]);
            return;
        case O_LAYERNORM:
            if ((n != 1 && n != 3) || !is_t(*a[0]) || (n == 3 && (!is_t(*a[1]) || !is_t(*a[2]))))
                no_impl(op, name, a, n);
            device_of(a, n);
            out.push_back(*a[0]);
            return;
        case O_TRANSPOSE: {
            if (n != 1 || !is_t(*a[0])) no_impl(op, name, a, n);
            const Value &x = *a[0];
            if (!x.known) {
                out.push_back(x);
                return;
            }
            int rk = x.shape.rank;
            if (!at.get_ints("perm", ints, false))
                for (int i = rk - 1; i >= 0; --i) ints.push_back(i);
            if ((int)ints.size() != rk) throw_fail(DSIM_EINVAL, "Transpose perm %s for rank %d", show_list(ints).c_str(), rk);
            bool seen[kMaxRank] = {};
            Shape r;
            for (int64_t p : ints) {
                int k = norm_axis(p, rk, "Transpose");
                if (seen[k]) throw_fail(DSIM_EINVAL, "Transpose perm %s is not a permutation", show_list(ints).c_str());
                seen[k] = true;
                r.push(x.shape.d[k]);
            }
            out.push_back(tensor(x.dt, &r, x.dev));
            return;
        }
        case O_FLATTEN: {
            if (n != 1 || !is_t(*a[0])) no_impl(op, name, a, n);
            const Value &x = *a[0];
            if (!x.known) {
                out.push_back(x);
                return;
            }
            int64_t ax = at.get_int("axis", 1);
            int64_t k = ax < 0 ? ax + x.shape.rank : ax;
            if (k < 0 || k > x.shape.rank) throw_fail(DSIM_EINVAL, "Flatten axis %lld out of range", (long long)ax);
            Shape r;
            r.push(prod(x.shape, 0, (int)k));
            r.push(prod(x.shape, (int)k, x.shape.rank));
            out.push_back(tensor(x.dt, &r, x.dev));
            return;
        }
        case O_SPLIT: {
            if (n != 1 || !is_t(*a[0])) no_impl(op, name, a, n);
            const Value &x = *a[0];
            at.get_ints("split", ints, true);
            if (ints.empty() || ints.size() > (size_t)kMaxOut) throw_fail(DSIM_EINVAL, "Split into %zu parts", ints.size());
            int64_t ax = at.get_int("axis", 0);
            if (!x.known) {
                for (size_t i = 0; i < ints.size(); ++i) out.push_back(tensor(x.dt, nullptr, x.dev));
                return;
            }
            int k = norm_axis(ax, x.shape.rank, "Split");
            int64_t sum = 0;
            for (int64_t p : ints) {
                if (p < 0) throw_fail(DSIM_EINVAL, "a negative Split part");
                if (__builtin_add_overflow(sum, p, &sum)) sum = -1;
            }
            if (sum != x.shape.d[k])
                throw_fail(DSIM_EINVAL, "split %s does not cover dimension %lld", show_list(ints).c_str(),
                      (long long)x.shape.d[k]);
            for (int64_t p : ints) {
                Shape r = x.shape;
                r.d[k] = p;
                out.push_back(tensor(x.dt, &r, x.dev));
            }
            return;
        }
        case O_MATMUL: {
            if (n != 2 || !is_t(*a[0]) || !is_t(*a[1])) no_impl(op, name, a, n);
            const Value &x = *a[0], &y = *a[1];
            int dev = device_of(a, 2);
            if (!x.known || !y.known) {
                out.push_back(tensor(x.dt, nullptr, dev));
                return;
            }
            const Shape &sa = x.shape, &sb = y.shape;
            if (sa.rank < 2 || sb.rank < 1 || sa.d[sa.rank - 1] != sb.d[sb.rank > 1 ? sb.rank - 2 : 0])
                throw_fail(DSIM_EINVAL, "MatMul of %s and %s", show_shape(sa).c_str(), show_shape(sb).c_str());
            Shape ba, bb, r;
            for (int i = 0; i < sa.rank - 2; ++i) ba.push(sa.d[i]);
            if (sb.rank > 1) {
                for (int i = 0; i < sb.rank - 2; ++i) bb.push(sb.d[i]);
                r = bcast(ba, bb);
            } else {
                r = ba;
            }
            r.push(sa.d[sa.rank - 2]);
            if (sb.rank > 1) r.push(sb.d[sb.rank - 1]);
            out.push_back(tensor(x.dt, &r, dev));
            return;
        }
        case O_GEMM: {
            if ((n != 2 && n != 3)) no_impl(op, name, a, n);
            for (int i = 0; i < n; ++i)
                if (!is_t(*a[i])) no_impl(op, name, a, n);
            const Value &x = *a[0], &y = *a[1];
            int dev = device_of(a, n);
            if (!x.known || !y.known) {
                out.push_back(tensor(x.dt, nullptr, dev));
                return;
            }
            const Shape &sa = x.shape, &sb = y.shape;
            bool ta = at.get_int("transA", 0) != 0, tb = at.get_int("transB", 0) != 0;
            if (sa.rank != 2 || sb.rank != 2 || sa.d[ta ? 0 : 1] != sb.d[tb ? 1 : 0])
                throw_fail(DSIM_EINVAL, "Gemm of %s and %s", show_shape(sa).c_str(), show_shape(sb).c_str());
            Shape r;
            r.push(sa.d[ta ? 1 : 0]);
            r.push(sb.d[tb ? 0 : 1]);
            out.push_back(tensor(x.dt, &r, dev));
            return;
        }
        case O_SEND: {
            if (n != 1 || !is_t(*a[0])) no_impl(op, name, a, n);
            const Value &x = *a[0];
            int64_t to = at.get_int("device", 0, true);
            if (to < 0 || to > INT32_MAX) throw_fail(DSIM_EINVAL, "Send to device %lld", (long long)to);
            if (to == x.dev) throw_fail(DSIM_EINVAL, "Send to its own device %lld", (long long)to);
            Value v = x;
            v.dev = (int32_t)to;
            out.push_back(std::move(v));
            return;
        }
        case O_ALLREDUCE: {
            if (n < 1 || n > kMaxOut) no_impl(op, name, a, n);
            for (int i = 0; i < n; ++i)
                if (!is_t(*a[i])) no_impl(op, name, a, n);
            for (int i = 0; i < n; ++i)
                for (int j = 0; j < i; ++j)
                    if (a[i]->dev == a[j]->dev) {
                        std::string devs("[");
                        char b[16];
                        for (int k = 0; k < n; ++k) {
                            snprintf(b, sizeof b, "%s%d", k ? ", " : "", a[k]->dev);
                            devs += b;
                        }
                        throw_fail(DSIM_EINVAL, "AllReduce inputs must lie on distinct devices, got %s]", devs.c_str());
                    }
            for (int i = 1; i < n; ++i)
                if (a[i]->known != a[0]->known || (a[0]->known && !(a[i]->shape == a[0]->shape)))
                    throw_fail(DSIM_EINVAL, "AllReduce of tensors of different shapes");
            for (int i = 0; i < n; ++i) out.push_back(*a[i]);
            return;
        }
        default:
            no_impl(op, name, a, n);
        }
    }
};

// ---------------------------------------------------------------------------
// Program text
// ---------------------------------------------------------------------------
// split at commas outside brackets, parentheses and quotes
void split_top(std::string_view s, std::vector<std::string_view> &out)
{
    out.clear();
    int depth = 0;
    char quote = 0;
    size_t start = 0;
    for (size_t i = 0; i < s.size(); ++i) {
        char c = s[i];
        if (quote) {
            if (c == quote) quote = 0;
            continue;
        }
        if (c == '"' || c == '\'') quote = c;
        else if (c == '(' || c == '[') ++depth;
        else if (c == ')' || c == ']') --depth;
        else if (c == ',' && depth == 0) {
            out.push_back(trim(s.substr(start, i - start)));
            start = i + 1;
        }
    }
    std::string_view last = trim(s.substr(start));
    if (!last.empty() || !out.empty()) out.push_back(last);
}

bool is_var_char(char c) { return is_word(c) || c == '.'; }

bool is_var(std::string_view s)
{
    if (s.size() < 2 || s[0] != '%') return false;
    for (size_t i = 1; i < s.size(); ++i)
        if (!is_var_char(s[i])) return false;
    return true;
}

// Tensor[DTYPE, (d0, ...) or ??, DEVICE] | DTYPE | DTYPE[DEVICE]
Value parse_type(std::string_view t)
{
    t = trim(t);
    if (t.substr(0, 7) == "Tensor[" && t.back() == ']') {
        std::vector<std::string_view> f;
        split_top(t.substr(7, t.size() - 8), f);
        if (f.size() != 3) throw_fail(DSIM_EINVAL, "cannot read the type '%.*s'", (int)t.size(), t.data());
        int dt = dtype_of(f[0]);
        if (dt < 0) throw_fail(DSIM_EINVAL, "unknown element type %.*s", (int)f[0].size(), f[0].data());
        Lit dl = parse_lit_all(f[2]);
        if (dl.t != Lit::INT || dl.i < 0 || dl.i > INT32_MAX)
            throw_fail(DSIM_EINVAL, "a device must be an integer >= 0");
        if (f[1] == "??") return tensor(dt, nullptr, (int)dl.i);
        if (f[1].empty() || f[1][0] != '(') throw_fail(DSIM_EINVAL, "a shape must be (d0, ...) or ??");
        Lit sl = parse_lit_all(f[1]);
        Shape s;
        if (sl.t == Lit::INT) {
            s.push(sl.i);   // "(n)" reads as rank 1
        } else {
            for (const Lit &d : sl.items) {
                if (d.t != Lit::INT) throw_fail(DSIM_EINVAL, "a dimension must be an integer");
                s.push(d.i);
            }
        }
        for (int i = 0; i < s.rank; ++i)
            if (s.d[i] < 0) throw_fail(DSIM_EINVAL, "a negative dimension");
        numel(s);
        return tensor(dt, &s, (int)dl.i);
    }
    size_t br = t.find('[');
    std::string_view nm = br == std::string_view::npos ? t : trim(t.substr(0, br));
    int dt = dtype_of(nm);
    if (dt < 0) throw_fail(DSIM_EINVAL, "cannot read the type '%.*s'", (int)t.size(), t.data());
    if (br == std::string_view::npos) return scalar(dt, -1);
    if (t.back() != ']') throw_fail(DSIM_EINVAL, "cannot read the type '%.*s'", (int)t.size(), t.data());
    Lit dl = parse_lit_all(t.substr(br + 1, t.size() - br - 2));
    if (dl.t != Lit::INT || dl.i < 0 || dl.i > INT32_MAX) throw_fail(DSIM_EINVAL, "a device must be an integer >= 0");
    return scalar(dt, (int)dl.i);
}

// ---------------------------------------------------------------------------
// The interpreter (Algorithm 1), with lowering or printing attached
// ---------------------------------------------------------------------------
struct Storage {
    int32_t dev;
    uint64_t bytes;
    bool keep, resident;
};

struct Rec {
    uint8_t kind, cls;
    int32_t a, b;
    u128 flops, bytes;
    uint64_t k;         // reduction length of a matrix multiplication
    int32_t off, n_created, n_read;
};

u128 nbytes(const Value &v)
{
    if (!v.known) throw_fail(DSIM_EINVAL, "cannot simulate: the shape of a %s tensor is unknown", kDtName[v.dt]);
    u128 b = (u128)(uint64_t)numel(v.shape) * (u128)kDtSize[v.dt];
    if (b >> 63) throw_fail(DSIM_ERANGE, "a tensor of 2^63 bytes or more");
    return b;
}

bool exact_f32(u128 v)
{
    if (v == 0) return true;
    uint64_t hi = (uint64_t)(v >> 64), lo = (uint64_t)v;
    int hb = hi ? 127 - __builtin_clzll(hi) : 63 - __builtin_clzll(lo);
    int drop = hb - 23;
    return drop <= 0 || (v & (((u128)1 << drop) - 1)) == 0;
}

void print_number(std::string &o, const Value &v, int64_t k)
{
    char b[40];
    if (!v.flt()) {
        snprintf(b, sizeof b, "%lld", (long long)v.iv[(size_t)k]);
    } else {
        double f = v.fv[(size_t)k];
        if (std::isnan(f)) snprintf(b, sizeof b, "nan");
        else if (std::isinf(f)) snprintf(b, sizeof b, f < 0 ? "-inf" : "inf");
        else {
            snprintf(b, sizeof b, "%.17g", f);
            if (!strpbrk(b, ".e")) strcat(b, ".0");
        }
    }
    o += b;
}

void print_conc(std::string &o, const Value &v, int dim, int64_t &k)
{
    if (dim == v.shape.rank) {
        print_number(o, v, k++);
        return;
    }
    o += '[';
    for (int64_t i = 0; i < v.shape.d[dim]; ++i) {
        if (i) o += ", ";
        print_conc(o, v, dim + 1, k);
    }
    o += ']';
}

void print_value(std::string &o, const Value &v)
{
    if (is_c(v)) {
        int64_t k = 0;
        print_conc(o, v, 0, k);
    } else if (is_s(v)) {
        o += kDtName[v.dt];
    } else {
        o += "Tensor[";
        o += kDtName[v.dt];
        o += ", ";
        o += v.known ? show_shape(v.shape) : std::string("??");
        char b[16];
        if (v.dev < 0)
            o += ", None]";
        else {
            snprintf(b, sizeof b, ", %d]", v.dev);
            o += b;
        }
    }
}

struct Program {
    // interpretation state
    std::vector<Value> vals;
    std::unordered_map<std::string_view, int32_t> var;
    std::vector<std::string_view> names;       // per value, its variable
    std::unordered_map<std::string_view, Value> inputs;
    Evaluator ev;
    Attrs attrs;
    std::vector<Value> res;
    std::vector<const Value *> args;
    std::vector<int32_t> arg_ix;
    std::vector<std::string_view> parts, outs;

    // lowering state
    bool lowering = false;
    int32_t n_dev = 8;
    std::vector<int32_t> st_of;                // per value: storage, -1 = none
    std::vector<Storage> st;
    std::vector<Rec> recs;
    std::vector<int32_t> refs;                 // per record: created, then read storages
    std::vector<int32_t> last;
    int32_t max_dev = -1;

    // printing state
    std::string *text = nullptr;

    void reset()
    {
        vals.clear();
        var.clear();
        names.clear();
        inputs.clear();
        st_of.clear();
        st.clear();
        recs.clear();
        refs.clear();
        max_dev = -1;
    }

    int32_t new_storage(const Value &t, bool resident, bool keep)
    {
        if (t.dev < 0) throw_fail(DSIM_EINVAL, "a tensor on no device");
        if (t.dev >= n_dev) throw_fail(DSIM_ERANGE, "a device beyond n_dev = %d", n_dev);
        max_dev = std::max(max_dev, t.dev);
        st.push_back(Storage{t.dev, (uint64_t)nbytes(t), keep, resident});
        return (int32_t)st.size() - 1;
    }

    void define(std::string_view name, Value &&v, int32_t storage)
    {
        auto ins = var.emplace(name, (int32_t)vals.size());
        if (!ins.second) throw_fail(DSIM_EINVAL, "%.*s is defined twice", (int)name.size(), name.data());
        if (text) {
            *text += name;
            *text += " = ";
            print_value(*text, v);
            *text += '\n';
        }
        vals.push_back(std::move(v));
        names.push_back(name);
        st_of.push_back(storage);
    }

    void read_inputs(std::string_view in)
    {
        size_t p = 0;
        int line = 0;
        while (p < in.size()) {
            size_t e = in.find('\n', p);
            if (e == std::string_view::npos) e = in.size();
            std::string_view l = trim(in.substr(p, e - p));
            p = e + 1;
            ++line;
            if (l.empty()) continue;
            size_t k = 1;
            while (k < l.size() && is_var_char(l[k])) ++k;
            std::string_view name = l.substr(0, k);
            if (!is_var(name)) throw_fail(DSIM_EINVAL, "inputs line %d: a binding must start with a %%name", line);
            std::string_view rest = trim(l.substr(k));
            Value v;
            try {
                if (!rest.empty() && rest[0] == '=')
                    v = lit_value(parse_lit_all(rest.substr(1)));
                else if (!rest.empty() && rest[0] == ':')
                    v = parse_type(rest.substr(1));
                else
                    throw_fail(DSIM_EINVAL, "expected '= value' or ': type'");
            } catch (Failure &f) {
                char m[sizeof f.msg];
                snprintf(m, sizeof m, "inputs line %d: %s", line, f.msg);
                memcpy(f.msg, m, sizeof m);
                throw;
            }
            if (!inputs.emplace(name, std::move(v)).second)
                throw_fail(DSIM_EINVAL, "inputs line %d: %.*s bound twice", line, (int)name.size(), name.data());
        }
    }

    void header(std::string_view l, bool mixed)
    {
        size_t open = l.find('('), close = l.rfind(')');
        if (open == std::string_view::npos || close == std::string_view::npos || close < open ||
            !trim(l.substr(close + 1)).empty())
            throw_fail(DSIM_EINVAL, "a bad function header");
        std::string_view fname = trim(l.substr(4, open - 4));
        if (fname.empty()) throw_fail(DSIM_EINVAL, "a bad function header");
        for (char c : fname)
            if (!is_word(c)) throw_fail(DSIM_EINVAL, "a bad function header");
        std::vector<std::string_view> ps;
        split_top(l.substr(open + 1, close - open - 1), ps);
        size_t used = 0;
        for (std::string_view p : ps) {
            size_t colon = p.find(':');
            if (colon == std::string_view::npos) throw_fail(DSIM_EINVAL, "a parameter without a type");
            std::string_view name = trim(p.substr(0, colon));
            if (!is_var(name)) throw_fail(DSIM_EINVAL, "a parameter name must be a %%name");
            std::string_view typ = trim(p.substr(colon + 1));
            bool keep = false;
            if (typ.size() > 4 && typ.substr(typ.size() - 4) == "keep" && is_space(typ[typ.size() - 5])) {
                keep = true;
                typ = trim(typ.substr(0, typ.size() - 4));
            }
            Value decl = parse_type(typ);
            auto it = inputs.find(name);
            Value v;
            if (it != inputs.end()) {
                v = it->second;
                ++used;
            } else {
                v = decl;
            }
            if (!mixed) v = abstract_of(v, decl.dev);
            int32_t s = -1;
            if (lowering && is_t(v)) s = new_storage(v, true, keep);
            define(name, std::move(v), s);
        }
        if (used != inputs.size())
            for (auto &kv : inputs)
                if (!var.count(kv.first))
                    throw_fail(DSIM_EINVAL, "input %.*s is not a parameter", (int)kv.first.size(), kv.first.data());
    }

    void add_rec(int kind, int a, int b, int cls, u128 flops, u128 bytes, const int32_t *created, int nc,
                 const int32_t *read, int nr, uint64_t k = 0)
    {
        Rec r;
        r.k = k;
        r.kind = (uint8_t)kind;
        r.cls = (uint8_t)cls;
        r.a = a;
        r.b = b;
        r.flops = flops;
        r.bytes = bytes;
        r.off = (int32_t)refs.size();
        r.n_created = nc;
        r.n_read = nr;
        refs.insert(refs.end(), created, created + nc);
        refs.insert(refs.end(), read, read + nr);
        recs.push_back(r);
    }

    // the records of one interpreted op (mixed interpretation)
    void lower_op(int op, const Attrs &at, int first_res)
    {
        int n = (int)args.size(), nres = (int)res.size();
        // storages the op reads: those of its tensor arguments, ascending, once each
        int32_t read[64];
        std::vector<int32_t> read_big;
        int32_t *rd = read;
        if (n > 64) {
            read_big.resize((size_t)n);
            rd = read_big.data();
        }
        int nr = 0;
        for (int i = 0; i < n; ++i)
            if (is_t(*args[i])) rd[nr++] = st_of[(size_t)arg_ix[(size_t)i]];
        std::sort(rd, rd + nr);
        nr = (int)(std::unique(rd, rd + nr) - rd);
        if (op == O_SEND) {
            int32_t out = new_storage(res[0], false, false);
            st_of[(size_t)first_res] = out;
            add_rec(1, args[0]->dev, res[0].dev, 0, 0, nbytes(*args[0]), &out, 1, rd, nr);
            return;
        }
        if (op == O_ALLREDUCE) {
            uint32_t mask = 0;
            for (int i = 0; i < n; ++i) {
                if (args[i]->dev < 0 || args[i]->dev >= n_dev)
                    throw_fail(DSIM_ERANGE, "a device beyond n_dev = %d", n_dev);
                mask |= 1u << args[i]->dev;
                st_of[(size_t)(first_res + i)] = st_of[(size_t)arg_ix[(size_t)i]];   // in place
            }
            add_rec(2, 0, (int)mask, 0, 0, nbytes(*args[0]), nullptr, 0, rd, nr);
            return;
        }
        bool any_t = false;
        for (const Value &r : res) any_t = any_t || is_t(r);
        if (!any_t) return;   // host-side value arithmetic
        if (is_view(op)) {
            int src = -1;
            for (int i = 0; i < n && src < 0; ++i)
                if (is_t(*args[i])) src = arg_ix[(size_t)i];
            if (src < 0) throw_fail(DSIM_EINVAL, "%s of a value that holds no memory", kOpName[op]);
            for (int i = 0; i < nres; ++i) st_of[(size_t)(first_res + i)] = st_of[(size_t)src];
            return;
        }
        int dev = -2;
        bool several = false;
        for (int i = 0; i < n; ++i)
            if (is_t(*args[i])) {
                several = several || (dev != -2 && dev != args[i]->dev);
                dev = args[i]->dev;
            }
        for (const Value &r : res)
            if (is_t(r)) {
                several = several || (dev != -2 && dev != r.dev);
                dev = r.dev;
            }
        if (several || dev < 0) throw_fail(DSIM_EINVAL, "%s on several devices or none", kOpName[op]);
        u128 moved = 0;
        for (int i = 0; i < n; ++i)
            if (is_t(*args[i])) moved += nbytes(*args[i]);
        for (const Value &r : res)
            if (is_t(r)) moved += nbytes(r);
        u128 flops = 0;
        int cls = 0;
        uint64_t kred = 0;
        const Value &r0 = res[0];
        if (op == O_MATMUL || op == O_GEMM) {
            const Shape &sa = args[0]->shape;
            int64_t k = op == O_MATMUL ? sa.d[sa.rank - 1] : sa.d[at.get_int("transA", 0) ? 0 : 1];
            u128 m = (u128)(uint64_t)numel(r0.shape);
            flops = 2 * m * (u128)(uint64_t)k + (op == O_GEMM && n == 3 ? m : 0);
            cls = 1;
            kred = (uint64_t)k;
        } else if (kEltFlops[op] >= 0) {
            flops = (u128)kEltFlops[op] * (u128)(uint64_t)numel(r0.shape);
        } else if (op != O_TRANSPOSE && op != O_CONCAT && op != O_SPLIT && op != O_GATHER) {
            throw_fail(DSIM_EINVAL, "no cost function for %s", kOpName[op]);
        }
        int32_t created[64];
        std::vector<int32_t> created_big;
        int32_t *cr = created;
        if (nres > 64) {
            created_big.resize((size_t)nres);
            cr = created_big.data();
        }
        int nc = 0;
        for (int i = 0; i < nres; ++i)
            if (is_t(res[(size_t)i])) {
                int32_t s = new_storage(res[(size_t)i], false, false);
                st_of[(size_t)(first_res + i)] = s;
                cr[nc++] = s;
            }
        add_rec(0, dev, 0, cls, flops, moved, cr, nc, rd, nr, kred);
    }

    void statement(std::string_view l, bool mixed)
    {
        size_t eq = l.find('=');
        if (eq == std::string_view::npos) throw_fail(DSIM_EINVAL, "cannot parse the statement");
        split_top(l.substr(0, eq), outs);
        if (outs.empty()) throw_fail(DSIM_EINVAL, "cannot parse the statement");
        for (std::string_view o : outs)
            if (!is_var(o)) throw_fail(DSIM_EINVAL, "cannot parse the statement");
        std::string_view r = trim(l.substr(eq + 1));
        size_t k = 0;
        while (k < r.size() && is_word(r[k])) ++k;
        std::string_view opname = r.substr(0, k);
        if (opname.empty()) throw_fail(DSIM_EINVAL, "cannot parse the statement");
        r = trim(r.substr(k));
        attrs.a.clear();
        if (!r.empty() && r[0] == '[') {
            int depth = 0;
            char quote = 0;
            size_t i = 0;
            for (; i < r.size(); ++i) {
                char c = r[i];
                if (quote) {
                    if (c == quote) quote = 0;
                } else if (c == '"' || c == '\'') {
                    quote = c;
                } else if (c == '[' || c == '(') {
                    ++depth;
                } else if (c == ']' || c == ')') {
                    if (--depth == 0) break;
                }
            }
            if (i >= r.size()) throw_fail(DSIM_EINVAL, "unclosed attributes");
            split_top(r.substr(1, i - 1), parts);
            for (std::string_view item : parts) {
                size_t e = item.find('=');
                if (e == std::string_view::npos) throw_fail(DSIM_EINVAL, "an attribute without a value");
                std::string_view key = trim(item.substr(0, e));
                for (const Attr &x : attrs.a)
                    if (x.key == key) throw_fail(DSIM_EINVAL, "attribute %.*s given twice", (int)key.size(), key.data());
                attrs.a.push_back(Attr{key, parse_lit_all(item.substr(e + 1))});
            }
            r = trim(r.substr(i + 1));
        }
        if (r.size() < 2 || r[0] != '(' || r.back() != ')') throw_fail(DSIM_EINVAL, "cannot parse the statement");
        split_top(r.substr(1, r.size() - 2), parts);
        args.clear();
        arg_ix.clear();
        for (std::string_view p : parts) {
            auto it = var.find(p);
            if (it == var.end()) {
                if (!is_var(p)) throw_fail(DSIM_EINVAL, "an argument must be a %%name");
                throw_fail(DSIM_EINVAL, "%.*s is not defined", (int)p.size(), p.data());
            }
            arg_ix.push_back(it->second);
        }
        for (int32_t ix : arg_ix) args.push_back(&vals[(size_t)ix]);
        for (std::string_view o : outs)
            if (var.count(o)) throw_fail(DSIM_EINVAL, "%.*s is defined twice", (int)o.size(), o.data());
        int op = op_of(opname);
        if (op < 0) throw_fail(DSIM_EINVAL, "no implementation of %.*s", (int)opname.size(), opname.data());
        ev.run(op, opname, attrs, args.data(), (int)args.size(), res);
        if (res.size() != outs.size())
            throw_fail(DSIM_EINVAL, "%s gives %zu values, %zu names", kOpName[op], res.size(), outs.size());
        bool any_c = false;
        for (const Value &x : res) any_c = any_c || is_c(x);
        if (!mixed && any_c) {
            // concrete results take the type of a value on the device of the
            // op's abstract arguments
            std::vector<Value> av;
            std::vector<const Value *> ap;
            av.reserve(args.size());
            for (const Value *x : args) av.push_back(abstract_of(*x, -1));
            for (const Value &x : av) ap.push_back(&x);
            int dev = device_of(ap.data(), (int)ap.size());
            for (Value &x : res) x = abstract_of(x, dev);
        }
        int first = (int)vals.size();
        for (size_t i = 0; i < outs.size(); ++i) {
            // a value's storage is set by lower_op; define() only records it
            define(outs[i], Value(res[i]), -1);
        }
        if (lowering) {
            // arguments may have moved when vals grew
            args.clear();
            for (int32_t ix : arg_ix) args.push_back(&vals[(size_t)ix]);
            lower_op(op, attrs, first);
        }
    }

    void run(std::string_view text_in, std::string_view inputs_text, bool mixed)
    {
        read_inputs(inputs_text);
        bool seen = false;
        size_t p = 0;
        int line = 0;
        vals.reserve(text_in.size() / 24 + 16);
        while (p < text_in.size()) {
            size_t e = text_in.find('\n', p);
            if (e == std::string_view::npos) e = text_in.size();
            std::string_view l = text_in.substr(p, e - p);
            p = e + 1;
            ++line;
            size_t hash = l.find('#');
            if (hash != std::string_view::npos) l = l.substr(0, hash);
            l = trim(l);
            if (l.empty()) continue;
            try {
                if (l.substr(0, 4) == "func" && l.size() > 4 && (is_space(l[4]) || l[4] == '(')) {
                    if (seen) throw_fail(DSIM_EINVAL, "a second function header");
                    seen = true;
                    header(l, mixed);
                } else if (!seen) {
                    throw_fail(DSIM_EINVAL, "a statement before the function header");
                } else if (l.substr(0, 6) == "return" && (l.size() == 6 || is_space(l[6]))) {
                    continue;
                } else {
                    statement(l, mixed);
                }
            } catch (Failure &f) {
                char m[sizeof f.msg];
                snprintf(m, sizeof m, "line %d: %s", line, f.msg);
                memcpy(f.msg, m, sizeof m);
                throw;
            }
        }
        if (!seen) throw_fail(DSIM_EINVAL, "no function");
    }

    // per-record frees, then the table columns (or nothing if code is NULL)
    void finish(int32_t max_ops, int64_t n_prog, int64_t c, uint32_t *code, float *flops, float *bytes,
                uint32_t *alloc, uint32_t *freeb, uint32_t *mm_k, uint64_t *init_live)
    {
        last.assign(st.size(), -1);
        for (size_t i = 0; i < recs.size(); ++i) {
            const Rec &r = recs[i];
            for (int k = 0; k < r.n_created + r.n_read; ++k) last[(size_t)refs[(size_t)(r.off + k)]] = (int32_t)i;
        }
        uint64_t init[kMaxTableDev] = {};
        for (const Storage &s : st)
            if (s.resident && __builtin_add_overflow(init[s.dev], s.bytes, &init[s.dev]))
                throw_fail(DSIM_ERANGE, "resident bytes of device %d reach 2^64", s.dev);
        bool write = code != nullptr && (int64_t)recs.size() <= max_ops;
        for (size_t i = 0; i < recs.size(); ++i) {
            const Rec &r = recs[i];
            u128 al = 0, fr = 0;
            for (int k = 0; k < r.n_created + r.n_read; ++k) {
                int32_t s = refs[(size_t)(r.off + k)];
                if (k < r.n_created) al += st[(size_t)s].bytes;
                if (last[(size_t)s] != (int32_t)i || st[(size_t)s].keep) continue;
                if (r.kind == 1 && k < r.n_created) throw_fail(DSIM_EINVAL, "a received tensor nothing reads");
                if (r.kind != 2) fr += st[(size_t)s].bytes;
            }
            if (!exact_f32(r.flops) || !exact_f32(r.bytes) || (al >> 32) || (fr >> 32) || (r.k >> 32))
                throw_fail(DSIM_ERANGE, "op %zu does not fit the table format exactly", i);
            if (!write) continue;
            size_t at = (size_t)i * (size_t)n_prog + (size_t)c;
            code[at] = (uint32_t)r.kind | (uint32_t)r.a << 8 | (uint32_t)r.b << 16 | (uint32_t)r.cls << 24;
            flops[at] = (float)r.flops;
            bytes[at] = (float)r.bytes;
            alloc[at] = (uint32_t)al;
            freeb[at] = (uint32_t)fr;
            if (mm_k) mm_k[at] = (uint32_t)r.k;
        }
        if (!write) return;
        for (int64_t j = (int64_t)recs.size(); j < max_ops; ++j) {
            size_t at = (size_t)j * (size_t)n_prog + (size_t)c;
            code[at] = 0;
            flops[at] = 0.0f;
            bytes[at] = 0.0f;
            alloc[at] = 0;
            freeb[at] = 0;
            if (mm_k) mm_k[at] = 0;
        }
        for (int d = 0; d < n_dev; ++d) init_live[(size_t)c * (size_t)n_dev + (size_t)d] = init[d];
    }
};

// one worker's share of dsim_lower_programs: programs [lo, hi)
struct Work {
    int64_t lo, hi;
    int64_t failed = -1;          // first program that failed (not for ENOSPC)
    Failure fail_info{};
    int64_t nospace = -1;         // first program with more records than max_ops
    int32_t max_recs = 0, max_dev = -1;
};

void lower_range(const char *const *programs, const char *const *inputs, int32_t n_dev, int32_t max_ops,
                 int64_t n_prog, uint32_t *code, float *flops, float *bytes, uint32_t *alloc, uint32_t *freeb,
                 uint32_t *mm_k, uint32_t *n_ops, uint64_t *init_live, Work &w)
{
    Program pr;
    pr.lowering = true;
    pr.n_dev = n_dev;
    for (int64_t c = w.lo; c < w.hi; ++c) {
        pr.reset();
        try {
            pr.run(programs[c], inputs && inputs[c] ? inputs[c] : "", true);
            pr.finish(max_ops, n_prog, c, code, flops, bytes, alloc, freeb, mm_k, init_live);
        } catch (Failure &f) {
            w.failed = c;
            w.fail_info = f;
            return;
        } catch (std::bad_alloc &) {
            w.failed = c;
            w.fail_info.st = DSIM_ERANGE;
            snprintf(w.fail_info.msg, sizeof w.fail_info.msg, "out of host memory");
            return;
        }
        int64_t nrec = (int64_t)pr.recs.size();
        if (nrec > INT32_MAX) nrec = INT32_MAX;
        w.max_recs = std::max(w.max_recs, (int32_t)nrec);
        w.max_dev = std::max(w.max_dev, pr.max_dev);
        if (code && nrec > max_ops && w.nospace < 0) w.nospace = c;
        if (n_ops) n_ops[c] = nrec > max_ops ? 0u : (uint32_t)nrec;
    }
}

}  // namespace
}  // namespace dsim

using namespace dsim;

extern "C" DSIM_API dsim_status dsim_interpret_program(const char *program, const char *inputs, int32_t mixed,
                                                       char *out, size_t cap, size_t *out_len)
{
    if (!program) return fail(DSIM_EINVAL, "program is NULL");
    if (mixed != 0 && mixed != 1) return fail(DSIM_EINVAL, "mixed must be 0 or 1");
    if (cap > 0 && !out) return fail(DSIM_EINVAL, "out is NULL with cap > 0");
    std::string text;
    try {
        Program pr;
        pr.text = &text;
        pr.run(program, inputs ? inputs : "", mixed != 0);
    } catch (Failure &f) {
        return fail(f.st, "%s", f.msg);
    } catch (std::bad_alloc &) {
        return fail(DSIM_ERANGE, "out of host memory");
    }
    if (out_len) *out_len = text.size() + 1;
    if (text.size() + 1 > cap) return fail(DSIM_ENOSPC, "the state needs %zu bytes, cap is %zu", text.size() + 1, cap);
    memcpy(out, text.c_str(), text.size() + 1);
    return DSIM_OK;
}

extern "C" DSIM_API dsim_status dsim_lower_programs(const char *const *programs, const char *const *inputs,
                                                    int64_t n_prog, int32_t n_dev, int32_t max_ops,
                                                    uint32_t *code, float *flops, float *bytes,
                                                    uint32_t *alloc_bytes, uint32_t *free_bytes, uint32_t *mm_k,
                                                    uint32_t *n_ops, uint64_t *init_live, int32_t *max_ops_used,
                                                    int32_t *n_dev_used, int32_t n_threads)
{
    if (!programs && n_prog > 0) return fail(DSIM_EINVAL, "programs is NULL");
    if (n_prog < 0 || n_prog > kMaxLaneCand) return fail(DSIM_ERANGE, "n_prog must be 0..2^32 - 256");
    if (n_dev < 1 || n_dev > kMaxTableDev) return fail(DSIM_ERANGE, "n_dev must be 1..8");
    if (max_ops < 0) return fail(DSIM_EINVAL, "max_ops must be >= 0");
    int given = (code != nullptr) + (flops != nullptr) + (bytes != nullptr) + (alloc_bytes != nullptr) +
                (free_bytes != nullptr) + (n_ops != nullptr) + (init_live != nullptr);
    if (given != 0 && given != 7)
        return fail(DSIM_EINVAL, "give all of code, flops, bytes, alloc_bytes, free_bytes, n_ops and init_live, or none");
    if (given == 0 && mm_k) return fail(DSIM_EINVAL, "mm_k without the other arrays");
    for (int64_t c = 0; c < n_prog; ++c)
        if (!programs[c]) return fail(DSIM_EINVAL, "program %lld is NULL", (long long)c);
    int64_t nt = std::max<int64_t>(1, std::min<int64_t>({(int64_t)n_threads, n_prog, 256}));
    std::vector<Work> w((size_t)nt);
    for (int64_t t = 0; t < nt; ++t) {
        w[(size_t)t].lo = n_prog * t / nt;
        w[(size_t)t].hi = n_prog * (t + 1) / nt;
    }
    auto job = [&](int64_t t) {
        lower_range(programs, inputs, n_dev, max_ops, n_prog, code, flops, bytes, alloc_bytes, free_bytes, mm_k,
                    n_ops, init_live, w[(size_t)t]);
    };
    if (nt == 1) {
        job(0);
    } else {
        std::vector<std::thread> th;
        try {
            for (int64_t t = 1; t < nt; ++t) th.emplace_back(job, t);
        } catch (std::exception &) {
            for (std::thread &x : th) x.join();
            return fail(DSIM_ERANGE, "cannot start %lld threads", (long long)nt);
        }
        job(0);
        for (std::thread &x : th) x.join();
    }
    int32_t mx = 0, md = -1;
    for (const Work &x : w) {
        if (x.failed >= 0)
            return fail(x.fail_info.st, "program %lld: %s", (long long)x.failed, x.fail_info.msg);
        mx = std::max(mx, x.max_recs);
        md = std::max(md, x.max_dev);
    }
    if (max_ops_used) *max_ops_used = mx;
    if (n_dev_used) *n_dev_used = md + 1 > 0 ? md + 1 : 1;
    for (const Work &x : w)
        if (x.nospace >= 0)
            return fail(DSIM_ENOSPC, "program %lld needs more than max_ops = %d records (%d at most)",
                        (long long)x.nospace, max_ops, mx);
    return DSIM_OK;
}

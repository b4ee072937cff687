// Drives the program front end (dsim_interpret_program, dsim_lower_programs)
// over valid programs read from the files named on the command line and over
// deterministic mutations of them -- bytes replaced by characters of the
// grammar, deleted, inserted, lines truncated or duplicated, numbers replaced
// by extreme values, or (every other round) one number by a small one --
// built with AddressSanitizer and
// UndefinedBehaviorSanitizer, so any out-of-bounds access, leak or undefined
// arithmetic in the parser, the interpreter or the lowering is reported.
// Every valid input must lower; every call must return a status.  Test code
// only.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

#include "dsim.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64()
{
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
static size_t pick(size_t n) { return n ? (size_t)(next_u64() % n) : 0; }

static const char kChars[] = "%[](),=:#.-+0123456789 \n\"'?eEakxy_TFIS";
static const char *kWords[] = {"-1", "0", "9223372036854775807", "-9223372036854775808", "99999999999999999999",
                               "1e308", "nan", "inf", "??", "Tensor[", "[[", "]]", "keep", "%x", "()",
                               "Float32", "Int32", "4294967296", "65536", "[]", "[0, 0]", "(0,)"};

static const char *kSmall[] = {"1", "2", "3", "4", "6", "7", "16", "0"};

// one number replaced by a small one: mostly still a valid program, so the
// interpreter and the lowering run to the end on shapes nobody chose
static std::string mutate_mild(const std::string &s)
{
    std::string t = s;
    size_t b = t.find_first_of("0123456789", pick(t.size()));
    if (b == std::string::npos) return t;
    size_t e = t.find_first_not_of("0123456789", b);
    t.replace(b, (e == std::string::npos ? t.size() : e) - b, kSmall[pick(sizeof kSmall / sizeof *kSmall)]);
    return t;
}

static std::string mutate(const std::string &s)
{
    std::string t = s;
    int n = 1 + (int)pick(4);
    for (int k = 0; k < n && !t.empty(); ++k) {
        size_t at = pick(t.size());
        switch (pick(8)) {
        case 0: t[at] = kChars[pick(sizeof kChars - 1)]; break;
        case 1: t.erase(at, 1 + pick(8)); break;
        case 2: t.insert(at, 1, kChars[pick(sizeof kChars - 1)]); break;
        case 3: t.insert(at, kWords[pick(sizeof kWords / sizeof *kWords)]); break;
        case 4: {   // truncate a line
            size_t e = t.find('\n', at);
            if (e != std::string::npos) t.erase(at, e - at);
            break;
        }
        case 5: {   // duplicate a line
            size_t b = t.rfind('\n', at), e = t.find('\n', at);
            b = b == std::string::npos ? 0 : b + 1;
            if (e != std::string::npos) t.insert(e + 1, t.substr(b, e - b + 1));
            break;
        }
        case 6: {   // replace a number
            size_t b = t.find_first_of("0123456789", at);
            if (b != std::string::npos) {
                size_t e = t.find_first_not_of("0123456789", b);
                t.replace(b, (e == std::string::npos ? t.size() : e) - b, kWords[pick(8)]);
            }
            break;
        }
        default:
            t.resize(at);
            break;
        }
    }
    return t;
}

static int g_calls = 0, g_ok = 0;

// interpret both ways, then lower: sizing pass and a full pass
static int exercise(const std::string &prog, const std::string &inputs, bool must_lower)
{
    const char *p = prog.c_str(), *in = inputs.c_str();
    size_t need = 0;
    for (int mixed = 0; mixed < 2; ++mixed) {
        dsim_status st = dsim_interpret_program(p, in, mixed, nullptr, 0, &need);
        ++g_calls;
        if (st == DSIM_ENOSPC) {
            std::vector<char> buf(need);
            st = dsim_interpret_program(p, in, mixed, buf.data(), buf.size(), &need);
            if (st != DSIM_OK || std::strlen(buf.data()) + 1 != need) {
                std::printf("interpret: size query and write disagree\n");
                return 1;
            }
        }
    }
    int32_t used = 0, devs = 0;
    const char *progs[3] = {p, p, p};
    const char *ins[3] = {in, in, in};
    const char *const *insp = inputs.empty() && pick(2) ? nullptr : ins;
    dsim_status st = dsim_lower_programs(progs, insp, 3, 8, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                         nullptr, nullptr, &used, &devs, 1);
    ++g_calls;
    if (st != DSIM_OK) {
        if (must_lower) {
            std::printf("a valid program did not lower: %s\n", dsim_last_error());
            return 1;
        }
        return 0;
    }
    int32_t rows = used + (int32_t)pick(3);
    size_t cells = (size_t)rows * 3 + 1;
    std::vector<uint32_t> code(cells), alloc(cells), freeb(cells), mm_k(cells), n_ops(3);
    std::vector<float> flops(cells), bytes(cells);
    std::vector<uint64_t> init(3 * 8);
    st = dsim_lower_programs(progs, insp, 3, 8, rows, code.data(), flops.data(), bytes.data(), alloc.data(),
                             freeb.data(), pick(2) ? mm_k.data() : nullptr, n_ops.data(), init.data(), &used, &devs,
                             1 + (int32_t)pick(4));
    ++g_calls;
    if (st != DSIM_OK) {   // the sizing pass accepted the same programs
        std::printf("full pass failed after the sizing pass: %s\n", dsim_last_error());
        return 1;
    }
    ++g_ok;
    return 0;
}

int main(int argc, char **argv)
{
    std::vector<std::string> progs;
    for (int i = 1; i < argc; ++i) {
        std::ifstream f(argv[i]);
        std::stringstream ss;
        ss << f.rdbuf();
        progs.push_back(ss.str());
    }
    if (progs.empty()) {
        std::printf("no programs given\n");
        return 1;
    }
    int failures = 0;
    // programs with a %flat parameter take the Reshape target's first entry
    // as a concrete input
    auto inputs_of = [](const std::string &p) {
        return p.find("%flat") != std::string::npos ? std::string("%flat = [-1]") : std::string();
    };
    for (const std::string &p : progs) failures += exercise(p, inputs_of(p), true);
    const int rounds = 4000;
    for (int r = 0; r < rounds; ++r) {
        const std::string &base = progs[pick(progs.size())];
        std::string inputs = inputs_of(base);
        if (!inputs.empty() && pick(4) == 0) inputs = mutate(inputs);
        failures += exercise(r % 2 ? mutate(base) : mutate_mild(base), inputs, false);
    }
    // argument errors
    const char *one[1] = {progs[0].c_str()};
    int32_t used = 0, devs = 0;
    uint32_t u = 0;
    if (dsim_lower_programs(nullptr, nullptr, 1, 8, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                            nullptr, nullptr, &used, &devs, 1) != DSIM_EINVAL ||
        dsim_lower_programs(one, nullptr, 1, 9, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                            nullptr, &used, &devs, 1) != DSIM_ERANGE ||
        dsim_lower_programs(one, nullptr, 1, 8, -1, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                            nullptr, nullptr, &used, &devs, 1) != DSIM_EINVAL ||
        dsim_lower_programs(one, nullptr, 1, 8, 4, &u, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                            nullptr, &used, &devs, 1) != DSIM_EINVAL ||
        dsim_lower_programs(one, nullptr, 1, 8, 4, nullptr, nullptr, nullptr, nullptr, nullptr, &u, nullptr,
                            nullptr, &used, &devs, 1) != DSIM_EINVAL ||
        dsim_interpret_program(nullptr, nullptr, 1, nullptr, 0, nullptr) != DSIM_EINVAL ||
        dsim_interpret_program(one[0], nullptr, 2, nullptr, 0, nullptr) != DSIM_EINVAL) {
        std::printf("an argument error was not reported\n");
        ++failures;
    }
    std::printf("%d calls, %d mutated batches lowered, %d failures\n", g_calls, g_ok, failures);
    return failures != 0;
}

// Host-only driver of the C ABI's argument checks for the sanitizer build
// (address and undefined-behaviour sanitizers).  Reads one call per line from
// stdin -- the entry point's name, then its arguments in declaration order
// (pointers as integers, 0 for NULL; they are never dereferenced: calls that
// pass the checks reach launch stubs) -- and prints, per call, the returned
// status, whether a launch stub was reached, and gdn_last_error().
#include <cstdint>
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "gdn.h"

namespace gdn {
extern int g_stub_launches;
}

namespace {

void* ptr(const std::string& s) { return reinterpret_cast<void*>(static_cast<uintptr_t>(std::stoull(s))); }

}  // namespace

int main() {
    std::string line;
    while (std::getline(std::cin, line)) {
        std::istringstream in(line);
        std::string fn;
        in >> fn;
        std::vector<std::string> a;
        for (std::string t; in >> t;) a.push_back(t);
        auto P = [&](size_t i) { return ptr(a.at(i)); };
        auto I = [&](size_t i) { return std::stoi(a.at(i)); };
        auto F = [&](size_t i) { return std::stof(a.at(i)); };
        auto Z = [&](size_t i) { return static_cast<size_t>(std::stoull(a.at(i))); };
        const int before = gdn::g_stub_launches;
        long long st = 0;
        if (fn == "gdn_decode") {
            st = gdn_decode(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4), (float*)P(5), P(6), I(7),
                            I(8), I(9), I(10), I(11), F(12), P(13));
        } else if (fn == "gdn_decode_indexed") {
            st = gdn_decode_indexed(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4), (float*)P(5),
                                    (const int32_t*)P(6), P(7), I(8), I(9), I(10), I(11), I(12), I(13), F(14),
                                    P(15));
        } else if (fn == "gdn_prefill_workspace_size") {
            st = (long long)gdn_prefill_workspace_size(I(0), I(1), I(2), I(3), I(4), I(5));
        } else if (fn == "gdn_prefill_varlen") {
            st = gdn_prefill_varlen(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4),
                                    (const int32_t*)P(5), (const float*)P(6), (float*)P(7), P(8), I(9), I(10),
                                    I(11), I(12), I(13), I(14), I(15), F(16), P(17), Z(18), P(19));
        } else if (fn == "gdn_prefill_varlen_indexed") {
            st = gdn_prefill_varlen_indexed(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4),
                                            (const int32_t*)P(5), (float*)P(6), (const int32_t*)P(7), P(8),
                                            I(9), I(10), I(11), I(12), I(13), I(14), I(15), I(16), F(17), P(18),
                                            Z(19), P(20));
        } else if (fn == "gdn_decode_multitoken") {
            st = gdn_decode_multitoken(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4),
                                       (const int32_t*)P(5), (float*)P(6), P(7), I(8), I(9), I(10), I(11), I(12),
                                       I(13), F(14), P(15), Z(16), P(17));
        } else if (fn == "gdn_prefill_varlen_noalloc") {
            st = gdn_prefill_varlen_noalloc(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4),
                                            (const int32_t*)P(5), (const float*)P(6), (float*)P(7), P(8), I(9),
                                            I(10), I(11), I(12), I(13), I(14), I(15), F(16), P(17));
        } else if (fn == "gdn_decode_ex") {
            st = gdn_decode_ex(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4), (float*)P(5),
                               (const int32_t*)P(6), I(7), P(8), I(9), I(10), I(11), I(12), I(13), F(14), I(15),
                               P(16));
        } else if (fn == "gdn_prefill_varlen_ex") {
            st = gdn_prefill_varlen_ex(P(0), P(1), P(2), (const float*)P(3), (const float*)P(4),
                                       (const int32_t*)P(5), (const float*)P(6), (float*)P(7),
                                       (const int32_t*)P(8), I(9), P(10), I(11), I(12), I(13), I(14), I(15),
                                       I(16), I(17), F(18), I(19), P(20), Z(21), P(22));
        } else if (fn == "gdn_abi_version") {
            st = gdn_abi_version();
        } else {
            std::printf("unknown\t0\t%s\n", fn.c_str());
            continue;
        }
        std::printf("%lld\t%d\t%s\n", st, gdn::g_stub_launches - before, gdn_last_error());
    }
    return 0;
}

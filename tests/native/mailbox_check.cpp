// The cross-process mailbox (csrc/mailbox.cpp) under AddressSanitizer and
// UBSan: a parent and a forked child ping-pong messages of every payload
// size up to the slot size, with pauses that send either side's wait to
// sleep on the futex; then the argument checks.  Prints "mailbox cases: N".
#include <sys/wait.h>
#include <unistd.h>

#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/hoccl.h"

namespace hoccl {
void set_error_message(const char *) {}
}  // namespace hoccl

static int fails = 0;
#define CHECK(c)                                                      \
    do {                                                              \
        if (!(c)) {                                                   \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            ++fails;                                                  \
        }                                                             \
    } while (0)

static std::vector<unsigned char> message(unsigned k, size_t len) {
    std::vector<unsigned char> m(len);
    for (size_t i = 0; i < len; ++i) m[i] = (unsigned char)(k * 131 + i * 7);
    return m;
}

int main() {
    const size_t kSlot = 300;
    const unsigned kMsgs = 1500;
    const std::string name = "/hoccl-check-" + std::to_string(getpid());
    hoccl_mailbox_t *box = nullptr;
    CHECK(hoccl_mailbox_create(name.c_str(), 2, kSlot, &box) == HOCCL_OK);
    if (!box) return 1;
    const pid_t child = fork();
    if (child == 0) {
        hoccl_mailbox_t *mine = nullptr;
        if (hoccl_mailbox_open(name.c_str(), &mine) != HOCCL_OK) _exit(2);
        std::vector<unsigned char> buf(kSlot);
        for (unsigned k = 1; k <= kMsgs; ++k) {
            size_t len = 0;
            if (hoccl_mailbox_wait(mine, 0, k, 10000) != HOCCL_OK) _exit(3);
            if (hoccl_mailbox_read(mine, 0, buf.data(), buf.size(), &len) != HOCCL_OK) _exit(4);
            if (len != k % (kSlot + 1) || (len && memcmp(buf.data(), message(k, len).data(), len) != 0))
                _exit(5);
            if (k % 97 == 0) usleep(1500);
            if (hoccl_mailbox_post(mine, 1, k, buf.data(), len) != HOCCL_OK) _exit(6);
        }
        hoccl_mailbox_close(mine);
        _exit(0);
    }
    int cases = 0;
    std::vector<unsigned char> back(kSlot);
    for (unsigned k = 1; k <= kMsgs; ++k) {
        const auto m = message(k, k % (kSlot + 1));
        CHECK(hoccl_mailbox_post(box, 0, k, m.data(), m.size()) == HOCCL_OK);
        if (k % 89 == 0) usleep(1500);
        size_t len = 0;
        if (hoccl_mailbox_wait(box, 1, k, 10000) != HOCCL_OK) {  // the child has died
            CHECK(!"the child answered");
            break;
        }
        CHECK(hoccl_mailbox_read(box, 1, back.data(), back.size(), &len) == HOCCL_OK);
        CHECK(len == m.size() && (len == 0 || memcmp(back.data(), m.data(), len) == 0));
        ++cases;
    }
    int status = 0;
    waitpid(child, &status, 0);
    CHECK(WIFEXITED(status) && WEXITSTATUS(status) == 0);
    // argument checks
    unsigned char big[kSlot + 1] = {};
    size_t len = 0;
    CHECK(hoccl_mailbox_post(box, 2, 1, big, 1) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_post(box, 0, 1, big, kSlot + 1) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_post(box, 0, 1, nullptr, 1) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_wait(box, 2, 1, 0) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_wait(box, 0, kMsgs + 1, 5) == HOCCL_ERR_TIMEOUT);
    CHECK(hoccl_mailbox_read(box, 1, big, 2, &len) == HOCCL_ERR_INVALID_ARG);  // last payload was longer
    CHECK(hoccl_mailbox_read(box, 0, nullptr, 0, nullptr) == HOCCL_ERR_INVALID_ARG);
    hoccl_mailbox_t *dup = nullptr;
    CHECK(hoccl_mailbox_create(name.c_str(), 2, kSlot, &dup) == HOCCL_ERR_INVALID_ARG && !dup);
    CHECK(hoccl_mailbox_unlink(name.c_str()) == HOCCL_OK);
    CHECK(hoccl_mailbox_open(name.c_str(), &dup) == HOCCL_ERR_INVALID_ARG && !dup);
    CHECK(hoccl_mailbox_create("no-slash", 1, 8, &dup) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_create("/a/b", 1, 8, &dup) == HOCCL_ERR_INVALID_ARG);
    CHECK(hoccl_mailbox_close(nullptr) == HOCCL_OK);
    cases += 12;
    hoccl_mailbox_close(box);
    if (fails) return 1;
    printf("mailbox cases: %d\n", cases);
    return 0;
}

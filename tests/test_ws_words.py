"""Host checks of the workspace's call generations, tagged coordination words
and per-call error word (``csrc/ws_words.h``, compiled here with g++ on its
own).

A sort pass's workgroups publish words that other workgroups poll until the
word carries the current call's tag; the words are never cleared between
calls, so a word must never look current to a later call or pass.  The error
word must belong to one call only, so that one failure does not stop every
later step."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR_DIR = os.path.join(ROOT, "paper_2112_02752_amd", "csrc")

PROGRAM = r"""
#include <stdio.h>
#include <stdint.h>
#include "ws_words.h"
using namespace emb;
static int fails = 0;
#define CHECK(c) do { if (!(c)) { printf("FAIL line %d: %s\n", __LINE__, #c); ++fails; } } while (0)
int main() {
  // generations: never 0 (the value of a cleared word), period 2^32 - 1
  CHECK(next_gen(0u) == 1u);
  CHECK(next_gen(1u) == 2u);
  CHECK(next_gen(0xfffffffeu) == 0xffffffffu);
  CHECK(next_gen(0xffffffffu) == 1u);
  uint32_t g = 0xfffffff0u;
  for (int i = 0; i < 40; ++i) { g = next_gen(g); CHECK(g != 0u); }
  // a word carries its count intact for every count below 2^30
  const uint32_t counts[] = {0u, 1u, 4095u, 65536u, (1u << 30) - 1u};
  const uint32_t gens[] = {1u, 2u, 7u, 0x7fffffffu, 0x80000000u, 0xfffffffeu, 0xffffffffu};
  for (uint32_t gg : gens)
    for (uint32_t p = 0; p < 4; ++p)
      for (uint32_t c : counts) {
        const uint64_t t = word_tag(gg, p);
        const uint64_t w = word_make(t, c);
        CHECK(word_current(w, t));
        CHECK(word_count(w) == c);
        // the same word is stale for every other pass and for the next and
        // previous generations, and a cleared word is stale for every tag
        for (uint32_t q = 0; q < 4; ++q)
          if (q != p) CHECK(!word_current(w, word_tag(gg, q)));
        CHECK(!word_current(w, word_tag(next_gen(gg), p)));
        CHECK(!word_current(word_make(word_tag(next_gen(gg), p), c), t));
        CHECK(!word_current(0ull, t));
      }
  // generations walk 1 .. 2^32 - 1 cyclically: after s calls from g0 the
  // generation is ((g0 - 1 + s) mod (2^32 - 1)) + 1
  {
    const uint32_t g0 = 0xfffffff0u;
    uint32_t x = g0;
    for (uint64_t s = 1; s <= 100; ++s) {
      x = next_gen(x);
      CHECK(x == (uint32_t)(((uint64_t)g0 - 1ull + s) % 0xffffffffull + 1ull));
    }
  }
  // error word: bits belong to the call whose generation the word carries
  uint64_t e = 0;
  CHECK(err_bits_of(e, 1u) == 0u);
  e = err_word_with(e, 1u, 1u);
  CHECK(err_bits_of(e, 1u) == 1u);
  e = err_word_with(e, 1u, 2u);
  CHECK(err_bits_of(e, 1u) == 3u);
  CHECK(err_bits_of(e, 2u) == 0u);           // the next call starts clean
  e = err_word_with(e, 2u, 4u);              // and replaces the old bits
  CHECK(err_bits_of(e, 2u) == 4u);
  CHECK(err_bits_of(e, 1u) == 0u);
  e = err_word_with(e, 0xffffffffu, 1u);
  CHECK(err_bits_of(e, 0xffffffffu) == 1u);
  CHECK(err_bits_of(e, next_gen(0xffffffffu)) == 0u);
  printf(fails ? "FAILED %d\n" : "ok\n", fails);
  return fails ? 1 : 0;
}
"""


@pytest.fixture(scope="module")
def program(tmp_path_factory):
    d = tmp_path_factory.mktemp("ws_words")
    src = d / "t.cpp"
    exe = d / "t"
    src.write_text(PROGRAM)
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-Wno-unused-variable",
                           "-I", HDR_DIR, str(src), "-o",
                           str(exe)])
    return str(exe)


def test_tag_and_error_word_arithmetic(program):
    r = subprocess.run([program], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"


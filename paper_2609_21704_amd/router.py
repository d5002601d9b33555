"""Prompt-complexity routing (SS III-B): which variant serves a request.

The router scores a prompt on the three features of SS III-B.1 and maps the
score to one of three classes (SS III-B.2):

    low       -> "int4": speculative decoding with the INT4 draft (Q4)
    moderate  -> "fp8":  speculative decoding with the FP8 draft (Q8)
    high      -> "f16":  direct decoding with the FP16 parent (Q16, SS III-D.5)

The paper names the features but gives neither their formulas nor the class
thresholds, so every number below is a stated reading:

  tokens    the prompt's length in tokens.
  syntax    sentence structure and depth: the mean over sentences of
            log2(words in the sentence) plus the sentence's clause depth
            (subordinating words and relative pronouns, one each; a comma,
            semicolon or colon, one half each; the deepest bracket nesting).
  entities  named-entity density: the share of words that look like names or
            terms (capitalised words that do not open a sentence, acronyms,
            words holding a digit, inner capitals or inner dots).

  score = 1/3 (log2(1 + tokens / 16) / log2(1 + 512 / 16)
               + syntax / 8 + entities / 0.3)

Each term is about 1 for a 512-token prompt, for sentences of ~20 words with
four clauses, and for a prompt where three words in ten are names.  Prompts of
at least `long_tokens` tokens are high whatever their score (the paper sends
long-context inputs to full precision).  `calibrate` sets the two thresholds
from a prompt set so that the classes take given shares of it; the default
shares are the class mix the paper reports over its benchmarks (28 % low,
52 % moderate, 20 % high, SS IV).
"""
from __future__ import annotations

import math
import re
from dataclasses import dataclass

ROUTES = ("int4", "fp8", "f16")
PAPER_MIX = (0.28, 0.52, 0.20)

_WORD = re.compile(r"[A-Za-z0-9]+(?:[.'_-][A-Za-z0-9]+)*")
_SENT_END = re.compile(r"(?<=[.!?])\s+|\n+")
_SUBORDINATORS = frozenset((
    "after", "although", "as", "because", "before", "if", "once", "since", "that", "though", "unless", "until",
    "when", "whenever", "where", "whereas", "wherever", "whether", "which", "while", "who", "whom", "whose"))
_PIECE = 6  # characters per token piece of the hashing tokenizer


@dataclass(frozen=True)
class Features:
    tokens: int
    syntax: float
    entities: float


def hash_tokenize(text: str, vocab: int) -> list[int]:
    """Token ids of a text: words and punctuation marks, each word cut into
    pieces of at most six characters, each piece hashed (FNV-1a, 32 bit) into
    [0, vocab).  A deterministic stand-in for a trained tokenizer, with a
    similar count of tokens per word (about 1.3 on plain text)."""
    ids = []
    for m in re.finditer(r"\w+|[^\w\s]", text):
        w = m.group(0)
        for i in range(0, len(w), _PIECE):
            h = 0x811C9DC5
            for b in w[i:i + _PIECE].encode():
                h = ((h ^ b) * 0x01000193) & 0xFFFFFFFF
            ids.append(h % vocab)
    return ids


def _bracket_depth(s: str) -> int:
    d = best = 0
    for ch in s:
        if ch in "([{":
            d += 1
            best = max(best, d)
        elif ch in ")]}" and d > 0:
            d -= 1
    return best


def _entity_like(word: str, opens_sentence: bool) -> bool:
    if any(ch.isdigit() for ch in word):
        return True
    if len(word) >= 2 and word.isupper():
        return True
    if any(ch.isupper() for ch in word[1:]) or "." in word or "_" in word:
        return True
    return word[0].isupper() and not opens_sentence


def features(text: str, tokens: int | None = None, vocab: int = 151936) -> Features:
    """The three features of a prompt (the module docstring defines them).
    `tokens` is the prompt's length when the caller has already tokenized it."""
    n_tok = len(hash_tokenize(text, vocab)) if tokens is None else int(tokens)
    sentences = [s for s in _SENT_END.split(text.strip()) if _WORD.search(s)]
    syn, words, ents = 0.0, 0, 0
    for s in sentences:
        ws = _WORD.findall(s)
        depth = sum(w.lower() in _SUBORDINATORS for w in ws)
        depth += 0.5 * sum(s.count(ch) for ch in ",;:") + _bracket_depth(s)
        syn += math.log2(len(ws)) + depth
        words += len(ws)
        ents += sum(_entity_like(w, i == 0) for i, w in enumerate(ws))
    return Features(tokens=n_tok, syntax=syn / len(sentences) if sentences else 0.0,
                    entities=ents / words if words else 0.0)


def score(f: Features) -> float:
    length = math.log2(1.0 + f.tokens / 16.0) / math.log2(1.0 + 512.0 / 16.0)
    return (length + f.syntax / 8.0 + f.entities / 0.3) / 3.0


class Router:
    """Scores prompts and picks their route (one of ROUTES)."""

    # Defaults: the thresholds `calibrate` gives on 2000 prompts of
    # synth.prompt_texts (seed 5) with the paper's mix, rounded.
    def __init__(self, low: float = 0.22, high: float = 0.53, long_tokens: int = 1024):
        if not low <= high:
            raise ValueError("thresholds must satisfy low <= high")
        self.low, self.high, self.long_tokens = float(low), float(high), int(long_tokens)

    def classify(self, f: Features) -> str:
        if f.tokens >= self.long_tokens:
            return "f16"
        s = score(f)
        return "int4" if s < self.low else ("fp8" if s < self.high else "f16")

    def route(self, text: str, tokens: int | None = None) -> str:
        return self.classify(features(text, tokens))

    def calibrate(self, texts, shares=PAPER_MIX) -> "Router":
        """Set the thresholds to the score quantiles that give the classes the
        shares (low, moderate, high) of `texts`; returns self."""
        if len(shares) != 3 or min(shares) < 0 or abs(sum(shares) - 1.0) > 1e-9:
            raise ValueError("shares must be three non-negative fractions summing to 1")
        scores = sorted(score(features(t)) for t in texts)
        if not scores:
            raise ValueError("calibration needs at least one prompt")

        def cut(frac):
            i = round(frac * len(scores))
            if i <= 0:
                return scores[0]
            if i >= len(scores):
                return math.nextafter(scores[-1], math.inf)
            return 0.5 * (scores[i - 1] + scores[i])

        self.low, self.high = cut(shares[0]), cut(shares[0] + shares[1])
        return self

"""Seeded synthetic text in the shapes of the paper's workloads.

The paper measures on real agent transcripts and web text that are not
available here (Sec. 5.4, Table tab:coldhead; the workload study in Sec. 2).
These generators stand in for them: prose built from a synthetic lexicon,
code-like lines, JSON tool outputs, log lines with timestamps and hex IDs,
and, for the multilingual configuration, accented Latin, Cyrillic, CJK runs
and emoji.  Every draw comes from ``random.Random`` seeded with a fixed
integer, so the same call always returns the same string.

Nothing in this module tokenizes, matches or merges: it only produces text.

Configurations (character counts are Unicode scalar values):

====  ===========  ==========  =======  ======  ============================
 k     chars        pattern     merges   train   style
====  ===========  ==========  =======  ======  ============================
 1     10,000       gpt2        1,024    200K    ASCII prose
 2     100,000      gpt2        8,192    2M      60% prose / 40% code
 3     1,000,000    gpt2        50,000   20M     agent transcript
 4     1,000,000    cl100k      100,000  20M     transcript, 20% multibyte
 5     3,000,000    cl100k      100,000  (k=4)   stress runs + 64x16,384 batch
====  ===========  ==========  =======  ======  ============================
"""

from __future__ import annotations

import bisect
import math
import random

__all__ = [
    "CONFIGS",
    "config_text",
    "training_text",
    "batch_docs",
    "latency_sample",
    "stress_text",
    "lexicon",
]

SEED_REQUEST = 0x5EED00
SEED_TRAIN = 0x7EA100
SEED_BATCH = 0x5EED50
SEED_LATENCY = 0x5EED80
SEED_LEXICON = 0x1E71C0

CONFIGS = {
    1: dict(name="c1", chars=10_000, pattern="gpt2", merges=1024, train_chars=200_000, style="prose"),
    2: dict(name="c2", chars=100_000, pattern="gpt2", merges=8192, train_chars=2_000_000, style="prose_code"),
    3: dict(name="c3", chars=1_000_000, pattern="gpt2", merges=50_000, train_chars=20_000_000, style="transcript"),
    4: dict(name="c4", chars=1_000_000, pattern="cl100k", merges=100_000, train_chars=20_000_000,
            style="transcript_mb"),
    5: dict(name="c5", chars=3_000_000, pattern="cl100k", merges=100_000, train_chars=None, style="stress",
            table_from=4, batch_docs=64, batch_doc_chars=16_384),
}

# ---------------------------------------------------------------------------
# lexicon
# ---------------------------------------------------------------------------

_ONSETS = ["", "", "b", "c", "d", "f", "g", "h", "j", "k", "l", "m", "n", "p", "r", "s", "t", "v", "w",
           "z", "br", "ch", "cl", "dr", "fl", "gr", "pl", "pr", "sh", "st", "str", "th", "tr", "sk", "sp",
           "qu", "bl", "cr", "fr", "gl", "sl", "sm", "sn", "sw", "tw", "wh", "kn", "ph", "sc"]
_NUCLEI = ["a", "e", "i", "o", "u", "a", "e", "i", "o", "y", "ai", "ea", "ee", "ie", "oa", "oo", "ou",
           "au", "io", "ue"]
_CODAS = ["", "", "", "", "n", "r", "s", "t", "l", "m", "d", "k", "ng", "nd", "st", "rt", "ck", "sh",
          "th", "x", "p", "ll", "ss", "nt", "rd", "mp", "lt", "ft"]

_LEX_CACHE: dict = {}


def lexicon(n_words: int = 2000):
    """2,000 unique lowercase words of 1-4 syllables, plus Zipf(s=1) cumulative weights."""
    if n_words in _LEX_CACHE:
        return _LEX_CACHE[n_words]
    rng = random.Random(SEED_LEXICON)
    seen = set()
    words = []
    while len(words) < n_words:
        n_syl = rng.choice((1, 1, 2, 2, 2, 3, 3, 4))
        w = "".join(rng.choice(_ONSETS) + rng.choice(_NUCLEI) + rng.choice(_CODAS) for _ in range(n_syl))
        if 2 <= len(w) <= 16 and w not in seen:
            seen.add(w)
            words.append(w)
    # frequent words are short, as in natural text: Zipf rank follows length
    words.sort(key=len)
    cum = []
    acc = 0.0
    for r in range(1, n_words + 1):
        acc += 1.0 / r
        cum.append(acc)
    _LEX_CACHE[n_words] = (words, cum)
    return words, cum


class _Source:
    """Random draws shared by all block writers of one text."""

    def __init__(self, seed: int, multibyte: float = 0.0):
        self.rng = random.Random(seed)
        self.words, self.cum = lexicon()
        self.total_w = self.cum[-1]
        # running tallies used to calibrate character shares
        self.n_chars = 0
        self.prose_chars = 0
        self.n_digits = 0
        self.n_punct = 0
        self.mb_target = multibyte
        self.n_mb = 0
        self.mb_kind = {"latin": 0, "cyr": 0, "cjk": 0, "emoji": 0}

    # -- lexicon words -------------------------------------------------------
    def word(self) -> str:
        i = bisect.bisect_left(self.cum, self.rng.random() * self.total_w)
        return self.words[min(i, len(self.words) - 1)]

    def ident(self) -> str:
        parts = [self.word() for _ in range(self.rng.choice((1, 2, 2, 3)))]
        if self.rng.random() < 0.5:
            return "_".join(parts)
        return parts[0] + "".join(p[:1].upper() + p[1:] for p in parts[1:])

    def number(self) -> str:
        n = self.rng.randint(1, 6)
        first = str(self.rng.randint(1, 9)) if n > 1 else str(self.rng.randint(0, 9))
        return first + "".join(str(self.rng.randint(0, 9)) for _ in range(n - 1))

    def hexid(self, lo=8, hi=32) -> str:
        return "".join(self.rng.choice("0123456789abcdef") for _ in range(self.rng.randint(lo, hi)))

    # -- multibyte substitution (transcript_mb only) --------------------------
    _ACCENTS = {
        "a": "áàâäãåāăą", "e": "éèêëēĕėęě", "i": "íìîïĩīĭį", "o": "óòôöõøōŏő", "u": "úùûüũūŭůűų",
        "c": "çćĉċč", "n": "ñńņňŉ", "s": "śŝşš", "z": "źżž", "l": "ĺļľŀł", "g": "ĝğġģ", "d": "ďđ",
        "r": "ŕŗř", "t": "ţťŧ", "y": "ýÿŷ", "h": "ĥħ", "k": "ķ", "w": "ŵ", "j": "ĵ",
    }
    _KIND_SHARE = {"latin": 0.30, "cyr": 0.30, "cjk": 0.35, "emoji": 0.05}

    def mb_wanted(self) -> bool:
        return self.mb_target > 0 and self.n_mb < self.mb_target * (self.n_chars + 8)

    def mb_word(self, base: str) -> str:
        """Return a multibyte replacement for ``base`` and account for it."""
        rng = self.rng
        tot = max(1, self.n_mb)
        kind = max(self._KIND_SHARE, key=lambda k: self._KIND_SHARE[k] - self.mb_kind[k] / tot)
        if kind == "latin":
            out = []
            n = 0
            for ch in base:
                acc = self._ACCENTS.get(ch)
                if acc and rng.random() < 0.6:
                    out.append(rng.choice(acc))
                    n += 1
                else:
                    out.append(ch)
            if n == 0:
                out.append(rng.choice(self._ACCENTS["e"]))
                n = 1
            s = "".join(out)
        elif kind == "cyr":
            n = rng.randint(3, 10)
            s = "".join(chr(rng.randint(0x430, 0x44F)) for _ in range(n))
            if rng.random() < 0.15:
                s = chr(ord(s[0]) - 0x20) + s[1:]
        elif kind == "cjk":
            n = rng.randint(4, 40)
            chars = []
            for i in range(n):
                chars.append(chr(rng.randint(0x4E00, 0x9FA5)))
                if i + 1 < n and rng.random() < 0.06:
                    chars.append(rng.choice("。，、"))
            s = "".join(chars)
            n = len(s)
        else:
            n = rng.randint(1, 3)
            s = "".join(chr(rng.randint(0x1F300, 0x1F64F)) for _ in range(n))
        self.n_mb += n
        self.mb_kind[kind] += n
        return s

    def emit(self, s: str) -> str:
        self.n_chars += len(s)
        return s


# ---------------------------------------------------------------------------
# block writers
# ---------------------------------------------------------------------------

_CONTRACTIONS = ["'s", "'t", "'re", "'ve", "'m", "'ll", "'d"]
_PUNCT_INNER = [",", ",", ",", ";", ":"]


def _sentence(src: _Source, mb: bool) -> str:
    rng = src.rng
    n = rng.randint(5, 25)
    toks = []
    for i in range(n):
        digit_short = src.n_digits < 0.05 * (src.prose_chars + 1)
        if digit_short and rng.random() < 0.5:
            w = src.number()
            src.n_digits += len(w)
        else:
            w = src.word()
            if i == 0 or rng.random() < 0.10:
                w = w[:1].upper() + w[1:]
            if mb and src.mb_wanted() and rng.random() < 0.8:
                w = src.mb_word(w)
        punct_short = src.n_punct < 0.05 * (src.prose_chars + 1)
        if punct_short and rng.random() < 0.5:
            r = rng.random()
            if r < 0.30:
                c = rng.choice(_CONTRACTIONS)
                w += c
                src.n_punct += 1
            elif r < 0.65 and i + 1 < n:
                w += rng.choice(_PUNCT_INNER)
                src.n_punct += 1
            elif r < 0.75:
                w = "(" + w + ")"
                src.n_punct += 2
            elif r < 0.85:
                w = '"' + w + '"'
                src.n_punct += 2
            else:
                w = w + "-" + src.word()
                src.n_punct += 1
        toks.append(w)
        src.n_chars += len(w) + 1
        src.prose_chars += len(w) + 1
    end = rng.choice((". ", ". ", ". ", "? ", "! "))
    src.n_punct += 1
    src.n_chars += 1
    src.prose_chars += 1
    return " ".join(toks) + end


def _prose(src: _Source, n_chars: int, mb: bool = False) -> str:
    out = []
    size = 0
    rng = src.rng
    para_left = rng.randint(3, 8)
    while size < n_chars:
        s = _sentence(src, mb)
        para_left -= 1
        if para_left == 0:
            s = s.rstrip(" ") + rng.choice(("\n", "\n\n"))
            para_left = rng.randint(3, 8)
        out.append(s)
        size += len(s)
    return "".join(out)


_OPS = ["=", "==", "!=", "<=", ">=", "+=", "->", "&&", "||", "+", "-", "*", "/"]


def _literal(src: _Source) -> str:
    rng = src.rng
    r = rng.random()
    if r < 0.4:
        return str(rng.randint(0, 99999))
    if r < 0.7:
        return "%d.%d" % (rng.randint(0, 999), rng.randint(0, 99999))
    if r < 0.85:
        return "0x" + src.hexid(2, 8)
    return "%d.%de%s%d" % (rng.randint(1, 9), rng.randint(0, 999), rng.choice(("-", "+", "")), rng.randint(1, 30))


def _expr(src: _Source, depth: int = 0) -> str:
    rng = src.rng
    r = rng.random()
    if r < 0.35 or depth > 2:
        return _literal(src) if rng.random() < 0.5 else src.ident()
    if r < 0.6:
        return "%s %s %s" % (_expr(src, depth + 1), rng.choice(_OPS[3:]), _expr(src, depth + 1))
    if r < 0.8:
        args = ", ".join(_expr(src, depth + 1) for _ in range(rng.randint(0, 3)))
        return "%s(%s)" % (src.ident(), args)
    if r < 0.9:
        return "%s[%s]" % (src.ident(), _expr(src, depth + 1))
    return "{%s}" % ", ".join(_expr(src, depth + 1) for _ in range(rng.randint(1, 3)))


def _code_block(src: _Source, n_lines: int) -> str:
    rng = src.rng
    unit = rng.choice((2, 4))
    depth = rng.randint(0, 2)
    lines = []
    for _ in range(n_lines):
        r = rng.random()
        ind = " " * (unit * depth)
        if r < 0.35:
            line = "%s%s %s %s" % (ind, src.ident(), rng.choice(("=", "+=", "=", ":=")), _expr(src))
            if rng.random() < 0.4:
                line += ";"
        elif r < 0.55:
            line = "%s%s(%s)" % (ind, src.ident(), ", ".join(_expr(src) for _ in range(rng.randint(0, 4))))
        elif r < 0.70:
            kw = rng.choice(("if", "for", "while", "elif", "def", "fn"))
            line = "%s%s (%s %s %s) {" % (ind, kw, src.ident(), rng.choice(_OPS[1:6]), _expr(src))
            depth = min(4, depth + 1)
        elif r < 0.80:
            line = ind + "}"
            depth = max(0, depth - 1)
        elif r < 0.92:
            cm = rng.choice(("#", "//"))
            line = "%s%s %s" % (ind, cm, " ".join(src.word() for _ in range(rng.randint(2, 10))))
        else:
            line = "%sreturn %s" % (ind, _expr(src))
        lines.append(line)
    s = "\n".join(lines) + "\n"
    src.n_chars += len(s)
    return s


def _code(src: _Source, n_chars: int) -> str:
    out = []
    size = 0
    while size < n_chars:
        b = _code_block(src, src.rng.randint(5, 40))
        out.append(b)
        size += len(b)
    return "".join(out)


def _json_value(src: _Source, depth: int, mb: bool):
    rng = src.rng
    r = rng.random()
    if depth < 4 and r < 0.25:
        return {"_".join(src.word() for _ in range(rng.randint(1, 3))): _json_value(src, depth + 1, mb)
                for _ in range(rng.randint(1, 5))}
    if depth < 4 and r < 0.35:
        return [_json_value(src, depth + 1, mb) for _ in range(rng.randint(0, 5))]
    if r < 0.55:
        return rng.randint(-100000, 10 ** rng.randint(1, 9))
    if r < 0.70:
        return round(rng.uniform(-1000, 1000), rng.randint(1, 6))
    if r < 0.75:
        return rng.choice((True, False, None))
    words = []
    for _ in range(rng.randint(1, 8)):
        w = src.word()
        if mb and src.mb_wanted() and rng.random() < 0.8:
            w = src.mb_word(w)
        words.append(w)
    if rng.random() < 0.15:
        words.append(src.hexid())
    return " ".join(words)


def _json_dump(v, ind: int, out: list):
    pad = "  " * ind
    if isinstance(v, dict):
        if not v:
            out.append("{}")
            return
        out.append("{\n")
        items = list(v.items())
        for i, (k, x) in enumerate(items):
            out.append('%s  "%s": ' % (pad, k))
            _json_dump(x, ind + 1, out)
            out.append(",\n" if i + 1 < len(items) else "\n")
        out.append(pad + "}")
    elif isinstance(v, list):
        if not v:
            out.append("[]")
            return
        out.append("[\n")
        for i, x in enumerate(v):
            out.append(pad + "  ")
            _json_dump(x, ind + 1, out)
            out.append(",\n" if i + 1 < len(v) else "\n")
        out.append(pad + "]")
    elif v is True:
        out.append("true")
    elif v is False:
        out.append("false")
    elif v is None:
        out.append("null")
    elif isinstance(v, str):
        out.append('"' + v.replace("\\", "\\\\").replace('"', '\\"') + '"')
    else:
        out.append(repr(v))


def _json_block(src: _Source, mb: bool) -> str:
    rng = src.rng
    obj = {"_".join(src.word() for _ in range(rng.randint(1, 2))): _json_value(src, 1, mb)
           for _ in range(rng.randint(2, 8))}
    out: list = []
    _json_dump(obj, 0, out)
    s = "".join(out) + "\n"
    src.n_chars += len(s)
    return s


def _log_block(src: _Source) -> str:
    rng = src.rng
    crlf = rng.random() < 0.10
    eol = "\r\n" if crlf else "\n"
    lines = []
    t = rng.randint(0, 86_000_000)
    for _ in range(rng.randint(5, 60)):
        t += rng.randint(1, 5000)
        hh, rem = divmod(t // 1000 % 86400, 3600)
        mm, ss = divmod(rem, 60)
        lvl = rng.choice(("INFO", "INFO", "INFO", "WARN", "ERROR", "DEBUG"))
        kv = " ".join("%s=%s" % (src.ident(), rng.choice((src.number(), src.hexid(4, 12), src.word())))
                      for _ in range(rng.randint(0, 4)))
        msg = " ".join(src.word() for _ in range(rng.randint(2, 9)))
        lines.append("2026-%02d-%02dT%02d:%02d:%02d.%03dZ %s [%s] %s id=%s %s" % (
            rng.randint(1, 12), rng.randint(1, 28), hh, mm, ss, t % 1000, lvl, src.ident(), msg,
            src.hexid(), kv))
    s = eol.join(lines) + eol
    src.n_chars += len(s)
    return s


def _transcript(src: _Source, n_chars: int, mb: bool) -> list:
    """Blocks of an agent session: prose turns, file dumps, JSON tool output, logs."""
    rng = src.rng
    blocks = []
    size = 0
    # block kinds are drawn so that each kind's share of the characters tracks
    # its target: prose turns 40%, file dumps 25%, JSON 20%, logs 15%
    share = {"prose": 0.40, "code": 0.25, "json": 0.20, "log": 0.15}
    got = {k: 0 for k in share}
    while size < n_chars:
        deficit = {k: share[k] * (size + 1) - got[k] + rng.random() * 3000 for k in share}
        kind = max(deficit, key=deficit.get)
        if kind == "prose":
            n = int(min(12_000, max(80, rng.lognormvariate(math.log(1400), 0.6))))
            b = _prose(src, n, mb)
        elif kind == "code":
            b = _code(src, rng.randint(2_000, 20_000))
        elif kind == "json":
            b = _json_block(src, mb)
        else:
            b = _log_block(src)
        b = b + "\n"
        blocks.append(b)
        got[kind] += len(b)
        size += len(b)
    return blocks


def _fit(blocks: list, n_chars: int) -> str:
    s = "".join(blocks)
    assert len(s) >= n_chars
    return s[:n_chars]


def _styled(style: str, seed: int, n_chars: int) -> str:
    if style == "prose":
        src = _Source(seed)
        return _fit([_prose(src, n_chars + 64)], n_chars)
    if style == "prose_code":
        src = _Source(seed)
        rng = src.rng
        blocks = []
        size = 0
        while size < n_chars + 64:
            if rng.random() < 0.6:
                b = _prose(src, rng.randint(300, 3000))
            else:
                b = _code_block(src, rng.randint(5, 40))
            b += "\n"
            blocks.append(b)
            size += len(b)
        return _fit(blocks, n_chars)
    if style == "transcript":
        src = _Source(seed)
        return _fit(_transcript(src, n_chars + 64, False), n_chars)
    if style == "transcript_mb":
        src = _Source(seed, multibyte=0.20)
        return _fit(_transcript(src, n_chars + 64, True), n_chars)
    if style == "stress":
        return stress_text(seed, n_chars)
    raise ValueError(style)


_LETTER_FREQ = [("e", 12.7), ("t", 9.1), ("a", 8.2), ("o", 7.5), ("i", 7.0), ("n", 6.7), ("s", 6.3),
                ("h", 6.1), ("r", 6.0), ("d", 4.3), ("l", 4.0), ("c", 2.8), ("u", 2.8), ("m", 2.4),
                ("w", 2.4), ("f", 2.2), ("g", 2.0), ("y", 2.0), ("p", 1.9), ("b", 1.5), ("v", 1.0),
                ("k", 0.8), ("j", 0.15), ("x", 0.15), ("q", 0.1), ("z", 0.07)]


def stress_text(seed: int, n_chars: int = 3_000_000) -> str:
    """Multilingual transcript filler with long degenerate runs inserted between blocks.

    Runs: 65,536 random letters (English letter frequencies); 32,768 chars of
    SP/TAB; 32,768 chars of LF, CRLF and SP; 25,000 each of 'a', '-', '=', '0';
    ten runs of 10,000 random digits.
    """
    rng = random.Random(seed ^ 0x51)
    letters = [c for c, _ in _LETTER_FREQ]
    lcum = []
    acc = 0.0
    for _, w in _LETTER_FREQ:
        acc += w
        lcum.append(acc)
    runs = []
    runs.append("".join(letters[min(bisect.bisect_left(lcum, rng.random() * acc), 25)] for _ in range(65_536)))
    runs.append("".join(rng.choice(" \t") for _ in range(32_768)))
    mixed = []
    m = 0
    while m < 32_768:
        t = rng.choice(("\n", "\r\n", " ", " "))
        if m + len(t) > 32_768:
            t = " "
        mixed.append(t)
        m += len(t)
    runs.append("".join(mixed))
    for c in "a-=0":
        runs.append(c * 25_000)
    for _ in range(10):
        runs.append("".join(rng.choice("0123456789") for _ in range(10_000)))
    special = sum(len(r) for r in runs)
    src = _Source(seed, multibyte=0.20)
    blocks = _transcript(src, n_chars - special + 64, True)
    filler = _fit(blocks, n_chars - special)
    # cut the filler at seeded positions and splice the runs in
    cuts = sorted(rng.randrange(1, len(filler)) for _ in runs)
    order = list(range(len(runs)))
    rng.shuffle(order)
    out = []
    prev = 0
    for c, i in zip(cuts, order):
        out.append(filler[prev:c])
        out.append(runs[i])
        prev = c
    out.append(filler[prev:])
    s = "".join(out)
    assert len(s) == n_chars
    return s


def config_text(k: int) -> str:
    """The seeded request text of configuration ``k`` (1..5)."""
    cfg = CONFIGS[k]
    return _styled(cfg["style"], SEED_REQUEST + k, cfg["chars"])


def training_text(k: int, n_chars: int | None = None) -> str:
    """The separate seeded sample the merge table of configuration ``k`` is trained on."""
    cfg = CONFIGS[k]
    if cfg.get("table_from"):
        raise ValueError("configuration %d reuses the table of configuration %d" % (k, cfg["table_from"]))
    n = cfg["train_chars"] if n_chars is None else n_chars
    return _styled(cfg["style"], SEED_TRAIN + k, n)


def batch_docs(n_docs: int = 64, doc_chars: int = 16_384) -> list:
    """The independent multilingual-transcript documents of the batch call."""
    return [_styled("transcript_mb", SEED_BATCH + j, doc_chars) for j in range(n_docs)]


def latency_sample(k: int, s: int) -> str:
    """Distinct 1M-char sample ``s`` (0..19) of configuration ``k`` (3 or 4) for latency percentiles."""
    cfg = CONFIGS[k]
    return _styled(cfg["style"], SEED_LATENCY + k * 32 + s, cfg["chars"])

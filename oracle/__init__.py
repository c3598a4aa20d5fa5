"""CPU oracle for exact GPT-family tokenization.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
definition that the HIP library is checked against.  Only the test-suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the library and
its Python binding never do, and this package never imports them.  The two
share no code: the only things both sides consume are the seeded texts of
``workloads`` and the merge tables stored there.

What it computes (the paper's output contract, Sec. 1 and the problem
statement of Sec. 3: the IDs of full reference tokenization of the request):

1. strict UTF-8 decoding (Python's decoder; invalid input is an error);
2. the class of every code point, from a table probed out of the regex engine
   the paper pins (``classes``);
3. leftmost-first regex pre-tokenization, written out by hand alternative by
   alternative for the GPT-2 and cl100k pattern families (``pretok``);
4. per-piece byte-level BPE that repeatedly merges the lowest-ranked adjacent
   pair, leftmost first (``bpe``), the model stage of the front-end/model
   factorisation (Appendix, Definition d:frontend, Lemma l:homo);
5. concatenation of the per-piece IDs (``tokenizer``).

``train`` is a small BPE trainer that produces merge tables from seeded text
(the paper uses frozen production tables; it never trains).  Parity of the
library does not depend on it, because both sides consume the same table.
"""

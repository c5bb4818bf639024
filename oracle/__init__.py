"""CPU oracle for the ReDASH garbled scaling gadget.

TEST INFRASTRUCTURE: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import, call, link or execute anything
under ``oracle/``.  The product path (``paper_2506_14489_amd``) must never
touch it and fails loudly when its HIP library is missing.

* ``rns``       -- value-level residue arithmetic (plain Python integers)
* ``oracle``    -- ctypes wrapper of ``gc_oracle.c`` (plain C: AES-128 from
                   FIPS-197, label hash, PRG, garble, encode, eval, decode)
* ``linear``    -- garbled dense and conv2d layers on LabelTensors (numpy):
                   Y = sum w X for the evaluator, Z = sum w Z - b R for the
                   garbler (Sec. 2.3 free operations)

The paper fixes no hash construction, label length, PRG, tweaks or packing;
those follow the construction stated in ``gc_oracle.c``.  They are pinned by
FIPS-197 (AES), by a step-by-step restatement on Python integers with
libcrypto's AES (fold, sigma, tweak words, feed-forward, digits, PRG
counters) and known-answer files, by the label invariants and decode results
the tests check, and by the independent HIP implementation.
"""

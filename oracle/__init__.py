"""CPU oracle for packed prefill (Prepacking, Zhao, Israel, Van den Broeck, Grover 2024).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the C-ABI library and its Python binding) never
does, and fails loudly when its HIP library is missing.

The oracle is a plain, slow, obviously-correct restatement of what the paper
defines, in float64 unless a caller asks for another precision:

* ``oracle.ffd``      -- BINPACK by first-fit decreasing (section 3.1), the
                         packed plan (TENSORIZE, RESTART-PE and the UNPACK
                         bookkeeping of Algorithm 1), the padded full-batching
                         plan (section 4.2) and a brute-force optimum for tiny
                         inputs;
* ``oracle.decoder``  -- the Llama-style decoder forward (section 2.1 and the
                         appendix model table), in three modes that the paper
                         claims agree exactly (section 3.3): every prompt
                         alone, packed rows under the literal independent mask
                         M' (section 3.2), and right-padded full batching;
                         and the greedy first token of every prompt;
* ``oracle.generate`` -- greedy generation after the prefill (sections 2.2
                         and 4.8) by full recomputation for every token, and
                         the teacher-forced rows a decode step must produce.

It shares no code with the HIP path; the only thing both sides share are the
seeded input generators in ``paper_2404_09529_amd.workloads``, which hold no
arithmetic of the method.

Parity status per function is listed in each module header.
"""

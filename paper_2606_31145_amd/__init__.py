"""SeKV decode-step library for MI355X (gfx950).

``paper_2606_31145_amd.sekv`` binds the HIP library (libsekv.so); importing it
raises if the library is not built.  ``paper_2606_31145_amd.accounting`` holds
the byte accounting of one decode step (pure Python).
"""

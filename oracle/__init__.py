"""Test-infrastructure oracle (fp64, CPU). Not part of the library's path."""
